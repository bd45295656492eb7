"""Benchmark of the emulated Trivance AllReduce on one MI355X.

python bench.py [--steps K] [--warmup W] [--workload NAME | --all] [--dtype f32|i32]
                [--no-cpu-baseline] [--no-summary]
python bench.py --sweep [--steps K] [--warmup W]     8..128 MiB per rank for every class
python bench.py --copy-probe BYTES                   a plain device copy (counter calibration)

A step is one whole emulated AllReduce (every pass of the schedule) over the workload's n rank
vectors, which are resident in HBM before timing starts. K steps are timed, bracketed by device
synchronisation; before each, the inputs are restored on the device (outside the events), so
every timed AllReduce works on the workload's own finite inputs. HIP events on the launch stream
bracket each step and, inside it, each phase (all passes of the latency-optimal variant; the
reduce-scatter and the all-gather), whose passes run back to back with one kernel family: group
time / launches is that family's average launch duration, used for the roofline. One more step after the timed region brackets every pass
with events (per-pass diagnostic only). Throughput counts the algorithmic
bytes of the step-by-step schedule (each participating location read once and each output
written once per pass; trivance_algorithmic_bytes).

Default workload: the largest single-GPU configuration, a 9 x 9 x 9 torus (729 virtual ranks),
bandwidth-optimal variant, 128 MiB of fp32 per rank (97.8 GB resident). Its line also summarises
the other configurations of the metric, measured in the same run (`other_configs`).
Prints one JSON line per workload.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2602_17254_amd import inputs  # noqa: E402

METRIC = "emulated AllReduce HBM GB/s and % of HBM peak, per-rank 8-128 MiB, 1 GPU"
HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, AMD published peak

# HBM traffic per launch measured with rocprofv3 --pmc (FETCH_SIZE / WRITE_SIZE, scaled by the
# same counters read for a plain copy of known size), keyed by workload and kernel, valid only for
# the kernel source it was measured on (sha256 of that source file, first 16 hex digits); the
# summaries are profiles/<kernel>_<workload>.md.
MEASURED_TRAFFIC = {
    ("ring243_B_32MiB", "block_step_kernel<reduce>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 3248038769},
    ("ring243_B_32MiB", "block_step_kernel<copy>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 2436096862},
    ("ring243_Bp_32MiB", "block_step_kernel<reduce>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 3248046986},
    ("ring243_Bp_32MiB", "block_step_kernel<copy>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 2436110148},
    ("torus27x27_B_4MiB", "block_step_kernel<reduce>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 1017880301},
    ("torus27x27_B_4MiB", "block_step_kernel<copy>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 763434309},
    ("torus27x27_Bp_4MiB", "block_step_kernel<reduce>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 1017886445},
    ("torus27x27_Bp_4MiB", "block_step_kernel<copy>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 763454489},
    ("torus9x9x9_B_128MiB", "block_step_kernel<reduce>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 32569005959},
    ("torus9x9x9_B_128MiB", "block_step_kernel<copy>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 24427297009},
    ("torus9x9x9_Bp_128MiB", "block_step_kernel<reduce>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 32568970997},
    ("torus9x9x9_Bp_128MiB", "block_step_kernel<copy>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 24427303559},
    ("ring81_L_8MiB", "latency_split_kernel"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 1358961457},
    ("ring64_L_8MiB", "slot_step_kernel"): {
        "src": "slot.hip", "src_sha": "2693a8a624b314e0", "bytes_per_launch": 3233243988},
    ("ring8_L_8MiB", "slot_step_kernel"): {
        "src": "slot.hip", "src_sha": "2693a8a624b314e0", "bytes_per_launch": 201398897},
    ("torus32x32_L_8MiB", "slot_step_kernel"): {
        "src": "slot.hip", "src_sha": "2693a8a624b314e0", "bytes_per_launch": 94333359694},
    ("ring64_B_8MiB", "tree_step_kernel<reduce>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 283157990},
    ("ring64_B_8MiB", "tree_step_kernel<copy>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 207665478},
    ("ring8_B_32MiB", "tree_step_kernel<reduce>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 251701844},
    ("ring8_B_32MiB", "tree_step_kernel<copy>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 184596997},
    ("torus16x16x16_B_8MiB", "tree_step_kernel<reduce>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 9723961811},
    ("torus16x16x16_B_8MiB", "tree_step_kernel<copy>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 6770476523},
    ("torus32x32_B_8MiB", "tree_step_kernel<reduce>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 2286938665},
    ("torus32x32_B_8MiB", "tree_step_kernel<copy>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 1679844735},
    ("torus8x64_B_8MiB", "tree_step_kernel<reduce>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 1550511409},
    ("torus8x64_B_8MiB", "tree_step_kernel<copy>"): {
        "src": "executor.hip", "src_sha": "4fae51c83bf720a1", "bytes_per_launch": 1132502565},
}


def phase_groups(phases):
    """[begin, end, phase] of every maximal run of consecutive passes with the same phase."""
    groups = []
    for p, ph in enumerate(phases):
        if groups and groups[-1][2] == ph:
            groups[-1][1] = p + 1
        else:
            groups.append([p, p + 1, ph])
    return groups


def _is_pow3(v):
    while v % 3 == 0:
        v //= 3
    return v == 1


def _src_sha(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def cpu_baseline(w, gpu_first_result_cols, cols, V_cols, seconds_target=10.0, max_runs=20):
    """Time the CPU oracle (as it stands, single-threaded numpy) on a column sample of the same
    workload, and compare its result with the GPU's first AllReduce on those columns. A sample
    that takes less than `seconds_target` is run again (same inputs, at most `max_runs` times in
    all) and the rate is taken over all runs."""
    from oracle import allreduce, partition, placement

    D = len(w.dims)
    if w.placement == "schedule":
        seg, blk = placement.column_labels(w.elems, w.dims, cols)
    else:
        seg, blk = partition.column_labels(w.elems, D, w.n, cols)
    def run():
        if w.variant == "L":
            return allreduce.allreduce(V_cols, w.dims, "L", col_seg=seg)
        return allreduce.allreduce(V_cols, w.dims, "B", col_seg=seg, col_blk=blk)

    t0 = time.perf_counter()
    out = run()
    runs = 1
    while time.perf_counter() - t0 < seconds_target and runs < max_runs:
        run()
        runs += 1
    dt = time.perf_counter() - t0
    # algorithmic bytes of the sample: the device path's own accounting, scaled to the sample
    import paper_2602_17254_amd as T

    ncols = len(cols)
    sample_bytes = T.trivance_algorithmic_bytes(T.trivance_plan(w.dims, w.variant, w.placement),
                                                w.elems) \
        * ncols / w.elems
    same = bool(np.array_equal(out, gpu_first_result_cols))
    if V_cols.dtype == np.int32:
        # integers: the exact column sums on every rank
        exact = {"gpu_exact_int_sum_on_sample": bool(np.array_equal(
            gpu_first_result_cols,
            np.broadcast_to(allreduce.exact_int_sum(V_cols), gpu_first_result_cols.shape)))}
    else:
        # the GPU's fp32 result on the sample against the fp64 sum: largest |error| / bound, where
        # the bound is 4 ceil(log3 n) 2^-23 sum|v|; below 1 means within the bound
        err = np.abs(gpu_first_result_cols.astype(np.float64) - allreduce.fp64_sum(V_cols)[None, :])
        bound = np.maximum(allreduce.fp32_error_bound(V_cols)[None, :], 1e-300)
        exact = {"gpu_fp64_bound_ratio_on_sample": round(float((err / bound).max()), 4)}
    import torch

    if w.congestion and torch.cuda.is_available():
        # the per-link message counts of the plan, GPU counter against the oracle's link walk
        from oracle import congestion

        got = T.trivance_congestion(T.trivance_plan(w.dims, w.variant, w.placement))
        exact["congestion_exact"] = bool(np.array_equal(got, congestion.link_loads(w.dims,
                                                                                  w.variant)))
    return {
        "value": round(sample_bytes * runs / dt / 1e9, 4),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "host": _host_cpu(),
        "sample": f"{ncols} of {w.elems} columns x {w.n} ranks (all passes), {runs} run(s), "
                  f"{dt:.2f} s",
        "seconds": round(dt, 3),
        "runs": runs,
        "matches_gpu_on_sample": same,
        **exact,
    }


def _host_cpu():
    """CPUs of the host the baseline ran on (the oracle itself uses one core)."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "os_cpu_count": os.cpu_count(),
            "affinity": len(os.sched_getaffinity(0))}


def _sample_for_baseline(w, budget_cols):
    rng = np.random.default_rng(w.seed + 99)
    if budget_cols >= w.elems:
        return np.arange(w.elems, dtype=np.int64)
    start = int(rng.integers(0, w.elems - budget_cols))
    return np.arange(start, start + budget_cols, dtype=np.int64)


def _inputs_on_device(w, dtype, device_rng=False):
    """The workload's inputs resident in HBM, and a function that restores them on a stream.

    dtype 'f32' or 'i32' (the workload's int32 companion). The counter-based U(-1, 1) inputs are
    regenerated in place on the device; host-generated inputs (numpy's N(0,1) and uniform int32,
    the workload's recipe) are uploaded once into a pristine device copy and restored from it with
    the library's streaming copy. With device_rng, N(0,1) and the int32 range come from torch's
    seeded device generator instead (same distributions, other values; used by the summary of
    the other configurations, which has no host-side oracle check).
    Returns (buf, regen, V_host); V_host is None when the values exist only on the device."""
    import torch

    import paper_2602_17254_amd as T

    shape = (w.n, w.elems)
    if dtype == "f32" and w.dist == "hash_uniform":
        buf = torch.empty(shape, dtype=torch.float32, device="cuda")
        return buf, (lambda s: T.trivance_fill_hash_uniform(buf, w.seed, s)), None
    V_host = None
    if device_rng:
        g = torch.Generator(device="cuda")
        g.manual_seed(w.seed if dtype == "f32" else w.int_seed)
        if dtype == "f32":
            pristine = torch.randn(shape, dtype=torch.float32, device="cuda", generator=g)
        else:
            lo, hi = w.int_range
            pristine = torch.randint(lo, hi + 1, shape, dtype=torch.int32, device="cuda",
                                     generator=g)
    else:
        if dtype == "f32":
            V_host = inputs.normal_f32(w.seed, w.n, w.elems)
        else:
            V_host = inputs.uniform_i32(w.int_seed, w.n, w.elems, *w.int_range)
        pristine = torch.from_numpy(V_host).cuda()
    buf = torch.empty_like(pristine)
    return buf, (lambda s: T.trivance_copy_device(buf, pristine, s)), V_host


def _all_finite(buf, rows=16):
    """True if no element of the float tensor is inf or NaN (checked a few rows at a time)."""
    import torch

    return all(bool(torch.isfinite(buf[r:r + rows]).all()) for r in range(0, buf.shape[0], rows))


def _workspace(plan, elems):
    """The device workspace a plan needs (None when it runs in place)."""
    import torch

    import paper_2602_17254_amd as T

    nbytes = T.trivance_workspace_bytes(plan, elems)
    return torch.empty(nbytes, dtype=torch.uint8, device="cuda") if nbytes else None


def _run_passes(buf, plan, ws, pb, pe, stream):
    import paper_2602_17254_amd as T

    if ws is None:
        T.trivance_allreduce_emulated_steps(buf, plan, pb, pe, stream)
    else:
        T.trivance_allreduce_emulated_steps_ws(buf, plan, ws, pb, pe, stream)


def _timed_steps(buf, plan, regen, groups, steps, stream, ws=None):
    """K AllReduces; before each, the inputs are restored (outside the events). Returns the
    per-step, per-phase-group event times (ms) and the wall time of the whole region (s)."""
    import torch

    G = len(groups)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(G + 1)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        regen(stream)
        ev[k][0].record(stream)
        for g, (pb, pe, _) in enumerate(groups):
            _run_passes(buf, plan, ws, pb, pe, stream)
            ev[k][g + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    group_ms = np.array([[ev[k][g].elapsed_time(ev[k][g + 1]) for g in range(G)]
                         for k in range(steps)])
    return group_ms, wall


def run_workload(w, steps, warmup, with_cpu, dtype="f32"):
    import torch

    import paper_2602_17254_amd as T

    torch.cuda.set_device(0)
    plan = T.trivance_plan(w.dims, w.variant, w.placement)
    P = plan.num_passes
    code = {"f32": T.F32, "i32": T.I32}[dtype]
    alg_bytes = T.trivance_algorithmic_bytes(plan, w.elems, code)
    pass_bytes = [T.trivance_pass_bytes(plan, w.elems, p, code) for p in range(P)]
    if dtype == "i32" and w.int_range is None:
        raise ValueError(f"{w.name} has no int32 input")

    # ---- inputs resident in HBM (untimed) ----
    _say(f"[bench] {w.name}: preparing inputs ({w.n} x {w.elems} {dtype})")
    buf, regen, V_host = _inputs_on_device(w, dtype)
    ws = _workspace(plan, w.elems)
    stream = torch.cuda.current_stream()

    # ---- first run: result kept for the CPU-baseline comparison ----
    # about 15 s of single-core oracle work: fewer columns as the rank count grows
    budget = {"L": 2_097_152, "B": min(60_000, (1 << 24) // w.n)}[w.variant]
    if w.variant == "L" and any(not _is_pow3(x) for x in w.dims):
        budget = min(budget, (1 << 22) // w.n)  # the oracle keeps several partials per rank
    cols = _sample_for_baseline(w, min(budget, w.elems))
    if V_host is not None:
        V_cols = np.ascontiguousarray(V_host[:, cols])
    else:
        V_cols = inputs.hash_uniform(w.seed, w.elems, np.arange(w.n), cols)
    del V_host
    regen(stream)
    _run_passes(buf, plan, ws, 0, P, stream)
    torch.cuda.synchronize()
    first_cols = None
    if with_cpu:
        first_cols = buf.index_select(1, torch.from_numpy(cols).cuda()).cpu().numpy()

    # ---- warmup (inputs restored before each AllReduce, like the timed steps) ----
    for _ in range(warmup):
        regen(stream)
        _run_passes(buf, plan, ws, 0, P, stream)
    torch.cuda.synchronize()

    # Passes of one phase run back to back with one kernel family (latency: every pass; reduce-
    # scatter; all-gather), so events at the phase boundaries give each family's average launch
    # duration (group time / launches) without a timing marker between every two kernels.
    groups = phase_groups([T.trivance_plan_step(plan, p)[0] for p in range(P)])

    # ---- timed region: K AllReduces on freshly restored inputs, events on the launch stream ----
    _say(f"[bench] {w.name}: timing {steps} steps x {P} passes")
    group_ms, wall = _timed_steps(buf, plan, regen, groups, steps, stream, ws)
    step_ms = group_ms.sum(axis=1)
    ms_per_step = float(step_ms.mean())
    value = alg_bytes / (ms_per_step * 1e-3) / 1e9
    finite = _all_finite(buf) if dtype == "f32" else True

    # ---- after the timed region: one diagnostic step with an event around every pass ----
    regen(stream)
    pev = [torch.cuda.Event(enable_timing=True) for _ in range(P + 1)]
    for p in range(P):
        pev[p].record(stream)
        _run_passes(buf, plan, ws, p, p + 1, stream)
    pev[P].record(stream)
    torch.cuda.synchronize()
    per_pass_ms = [pev[p].elapsed_time(pev[p + 1]) for p in range(P)]

    # dominant kernel: the family with the most time in the timed region
    tree = any(not _is_pow3(s) for s in w.dims)
    names = {0: "slot_step_kernel" if tree else "latency_split_kernel",
             1: "tree_step_kernel<reduce>" if tree else "block_step_kernel<reduce>",
             2: "tree_step_kernel<copy>" if tree else "block_step_kernel<copy>"}
    dg = int(np.argmax(group_ms.sum(axis=0)))
    pb, pe, dom = groups[dg]
    launches = pe - pb
    dom_ms = float(group_ms[:, dg].mean()) / launches
    dom_bytes = sum(pass_bytes[pb:pe]) / launches
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    # counters were taken on the fp32 runs
    meas = MEASURED_TRAFFIC.get((w.name, names[dom])) if dtype == "f32" else None
    traffic = None
    if meas and meas["src_sha"] == _src_sha(os.path.join(ROOT, "paper_2602_17254_amd", "csrc",
                                                          meas["src"])):
        traffic = meas["bytes_per_launch"]
    roofline = {
        "bound": "hbm",
        "kernel": names[dom],
        "achieved": round(achieved, 1),
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBPS, 4),
        "traffic": traffic,
        "alg_bytes_per_launch": int(dom_bytes),
        "avg_launch_ms": round(dom_ms, 4),
        "launches_per_step": launches,
    }
    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "topology": "x".join(map(str, w.dims)),
            "variant": {"L": "latency-optimal", "B": "bandwidth-optimal"}[w.variant],
            "block_placement": "schedule digits" if w.placement == "schedule" else "natural",
            "n_ranks": w.n,
            "elems_per_rank": w.elems,
            "rank_bytes": w.rank_bytes,
            "resident_bytes": w.n * w.rank_bytes,
            "passes": P,
            "alg_bytes_per_step": alg_bytes,
            "input": w.dist if dtype == "f32" else f"uniform int32 {w.int_range}",
        },
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBPS, 2),
        "timing": "ms_per_step = mean of the K event-timed AllReduces on the launch stream; the "
                  "inputs are restored before every AllReduce, outside the events",
        "step_ms_events": {"mean": round(ms_per_step, 4),
                           "median": round(float(np.median(step_ms)), 4),
                           "min": round(float(step_ms.min()), 4),
                           "max": round(float(step_ms.max()), 4)},
        "wall_ms_per_step_incl_input_restore": round(wall * 1e3 / steps, 4),
        "timed_outputs_finite": finite,
        "per_pass_ms_diagnostic": [round(float(x), 4) for x in per_pass_ms],
        "roofline": roofline,
        "cpu_baseline": None,
    }
    if ws is not None:
        line["config"]["workspace_bytes"] = ws.numel()
    del buf, regen, ws
    torch.cuda.empty_cache()
    ceiling = copy_ceiling()
    line["copy_ceiling"] = ceiling
    roofline["vs_copy_ceiling"] = round(achieved / ceiling["GBps"], 4)
    if with_cpu:
        _say(f"[bench] {w.name}: CPU oracle on {len(cols)} columns")
        line["cpu_baseline"] = cpu_baseline(w, first_cols, cols, V_cols)
    return line


# The other named configurations of the metric, summarised inside the headline line.
SUMMARY_JOBS = [("ring9_L_4KiB", "f32"), ("ring81_L_8MiB", "f32"), ("ring243_B_32MiB", "f32"),
                ("ring243_B_32MiB", "i32"), ("torus27x27_B_4MiB", "f32")]


def summary_line(w, dtype, steps=10, warmup=2, with_cpu=True):
    """Throughput of one more configuration in the same run, with inputs from torch's seeded
    device generator (the workload's distribution) restored before every timed AllReduce, and a
    check of the result on the device: int32 against the exact column sums, fp32 within
    4 ceil(log3 n) 2^-23 sum|v| of an fp64 sum. With with_cpu, the oracle is also timed on one
    core on a column sample of the same inputs (about 3 s) and compared with the GPU result on
    those columns (`cpu_baseline`)."""
    import torch

    import paper_2602_17254_amd as T

    plan = T.trivance_plan(w.dims, w.variant, w.placement)
    code = {"f32": T.F32, "i32": T.I32}[dtype]
    alg_bytes = T.trivance_algorithmic_bytes(plan, w.elems, code)
    steps_bound = 0
    while 3 ** steps_bound < w.n:  # ceil(log3 n)
        steps_bound += 1
    _say(f"[bench] summary {w.name} {dtype}")
    buf, regen, _ = _inputs_on_device(w, dtype, device_rng=True)
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        regen(stream)
        T.trivance_allreduce_emulated(buf, plan, stream)
    groups = phase_groups([T.trivance_plan_step(plan, p)[0] for p in range(plan.num_passes)])
    group_ms, _ = _timed_steps(buf, plan, regen, groups, steps, stream)
    ms = float(group_ms.sum(axis=1).mean())
    # result check on the last timed AllReduce: restore a copy of its inputs, compare column sums
    # over every column, a few rows at a time
    out = buf.clone()
    regen(stream)
    torch.cuda.synchronize()
    ok = True
    for e0 in range(0, w.elems, 1 << 20):
        e1 = min(w.elems, e0 + (1 << 20))
        if dtype == "i32":
            exact = buf[:, e0:e1].to(torch.int64).sum(0)
            exact = ((exact + 2 ** 31) % 2 ** 32 - 2 ** 31).to(torch.int32)
            ok = ok and bool((out[:, e0:e1] == exact[None, :]).all())
        else:
            x = buf[:, e0:e1].to(torch.float64)
            bound = 4.0 * steps_bound * 2.0 ** -23 * x.abs().sum(0)
            err = (out[:, e0:e1].to(torch.float64) - x.sum(0)[None, :]).abs()
            ok = ok and bool((err <= bound[None, :]).all())
    oracle = None
    if with_cpu:
        budget = {"L": 1 << 18, "B": min(12_000, (1 << 22) // w.n)}[w.variant]
        cols = _sample_for_baseline(w, min(budget, w.elems))
        idx = torch.from_numpy(cols).cuda()
        V_cols = buf.index_select(1, idx).cpu().numpy()
        got_cols = out.index_select(1, idx).cpu().numpy()
        oracle = cpu_baseline(w, got_cols, cols, V_cols, seconds_target=3.0, max_runs=10)
        oracle.pop("host", None)
    del buf, regen, out
    torch.cuda.empty_cache()
    gbps = alg_bytes / (ms * 1e-3) / 1e9
    return {"workload": w.name, "dtype": dtype, "ms_per_step": round(ms, 4),
            "GBps": round(gbps, 1), "pct_of_hbm_peak": round(100 * gbps / HBM_PEAK_GBPS, 2),
            "steps": steps, "input": "torch device generator, " +
            ("N(0,1)" if dtype == "f32" else f"uniform int32 {w.int_range}"),
            "result_check": ("exact column sums" if dtype == "i32" else
                             "within 4 ceil(log3 n) 2^-23 sum|v| of fp64"),
            "result_ok": ok, **({"cpu_baseline": oracle} if oracle else {})}


def copy_ceiling(nbytes: int = 1 << 30, reps: int = 10) -> dict:
    """The practical HBM ceiling in the same run: the library's plain streaming copy
    (trivance_copy_device, one 16-byte streaming load and store per lane) of `nbytes`, timed
    with HIP events on the stream it runs on. Bytes counted: read + written."""
    import torch

    import paper_2602_17254_amd as T

    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1.0)
    s = torch.cuda.current_stream()
    for _ in range(3):
        T.trivance_copy_device(dst, src, s)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(s)
    for _ in range(reps):
        T.trivance_copy_device(dst, src, s)
    e1.record(s)
    e1.synchronize()
    ms = e0.elapsed_time(e1) / reps
    gbps = 2 * nbytes / (ms * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return {"kernel": "copy_stream_kernel", "bytes_per_launch": 2 * nbytes,
            "avg_launch_ms": round(ms, 4), "GBps": round(gbps, 1),
            "frac_of_peak": round(gbps / HBM_PEAK_GBPS, 4)}


def copy_probe(nbytes: int, reps: int = 3) -> None:
    """A plain device copy of known size (torch's copy kernel), used to calibrate the rocprofv3
    FETCH_SIZE / WRITE_SIZE counters against known traffic. Prints one JSON line."""
    import torch

    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / reps
    print(json.dumps({"copy_probe_bytes": nbytes, "reps": reps, "ms": round(dt * 1e3, 4),
                      "GBps_read_plus_write": round(2 * nbytes / dt / 1e9, 1)}), flush=True)


SWEEP_CLASSES = [((81,), "L"), ((243,), "B"), ((27, 27), "B"), ((9, 9, 9), "B"), ((8,), "B"),
                 ((64,), "B"), ((32, 32), "B"), ((8, 64), "B"), ((16, 16, 16), "B"),
                 ((8,), "L"), ((64,), "L"), ((32, 32), "L")]
# the power-of-three bandwidth-optimal classes again with message-contiguous block placement
SWEEP_PLACED = [(243,), (27, 27), (9, 9, 9)]
SWEEP_MIB = [8, 16, 32, 64, 128]
# buffers plus workspace: 16x16x16 stops at 32 MiB per rank (128 GiB), the latency-optimal 32x32
# at 8 MiB (8 GiB of buffers and 144 GiB of partial sums)
SWEEP_MAX_RESIDENT = 160 * 2 ** 30


def sweep(steps: int, warmup: int) -> None:
    """Throughput of each topology/variant class at 8..128 MiB per rank (one JSON line each).
    Inputs are the device-generated U(-1, 1) values; correctness is covered by the test suite."""
    import torch

    import paper_2602_17254_amd as T

    torch.cuda.set_device(0)
    classes = [(d, v, "natural") for d, v in SWEEP_CLASSES] + \
              [(d, "B", "schedule") for d in SWEEP_PLACED]
    for dims, variant, placement in classes:
        plan = T.trivance_plan(dims, variant, placement)
        n = plan.n
        for mib in SWEEP_MIB:
            E = mib * 2 ** 20 // 4
            if n * E * 4 + T.trivance_workspace_bytes(plan, E) > SWEEP_MAX_RESIDENT:
                continue
            _say(f"[sweep] {'x'.join(map(str, dims))} {variant} {placement} {mib} MiB per rank")
            buf = torch.empty((n, E), dtype=torch.float32, device="cuda")
            ws = _workspace(plan, E)
            T.trivance_fill_hash_uniform(buf, 7)
            s0 = torch.cuda.current_stream()
            for _ in range(warmup):
                _run_passes(buf, plan, ws, 0, plan.num_passes, s0)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(steps):
                _run_passes(buf, plan, ws, 0, plan.num_passes, s0)
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t0) * 1e3 / steps
            alg = T.trivance_algorithmic_bytes(plan, E)
            gbps = alg / (ms * 1e-3) / 1e9
            print(json.dumps({"sweep": "x".join(map(str, dims)), "variant": variant,
                              "block_placement": placement, "rank_mib": mib, "n_ranks": n, "passes": plan.num_passes,
                              "ms_per_allreduce": round(ms, 4), "GBps": round(gbps, 1),
                              "pct_of_hbm_peak": round(100 * gbps / HBM_PEAK_GBPS, 2),
                              "resident_GB": round(n * E * 4 / 1e9, 2),
                              "workspace_GB": round(T.trivance_workspace_bytes(plan, E) / 1e9, 2)}),
                  flush=True)
            del buf, ws
            torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=inputs.HEADLINE, choices=sorted(inputs.WORKLOADS))
    ap.add_argument("--all", action="store_true", help="every named workload, one line each")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-summary", action="store_true",
                    help="skip the summary of the other configurations in the headline line")
    ap.add_argument("--dtype", default="f32", choices=["f32", "i32"],
                    help="element type (i32 needs a workload with an int32 input)")
    ap.add_argument("--sweep", action="store_true",
                    help="8..128 MiB per rank for every topology/variant class")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures a single-GPU emulation of all virtual ranks; it runs on exactly "
              "one GPU (--gpus 1).", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.sweep:
        sweep(args.steps, args.warmup)
        return
    if args.all:
        # every workload in fp32, plus the int32 companion of those that define one
        jobs = [(name, "f32") for name in inputs.WORKLOADS]
        jobs += [(name, "i32") for name, w in inputs.WORKLOADS.items() if w.int_range is not None]
    else:
        jobs = [(args.workload, args.dtype)]
    for name, dtype in jobs:
        line = run_workload(inputs.WORKLOADS[name], args.steps, args.warmup,
                            with_cpu=not args.no_cpu_baseline, dtype=dtype)
        if not args.all and not args.no_summary and name == inputs.HEADLINE:
            line["other_configs"] = [summary_line(inputs.WORKLOADS[n], d,
                                                  with_cpu=not args.no_cpu_baseline)
                                     for n, d in SUMMARY_JOBS]
        print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
