"""Thin ctypes binding of libtrivance.so (the C ABI declared in include/trivance.h).

Argument marshalling only: every step of the emulated AllReduce runs in the library's HIP
kernels. Functions keep the C names. PyTorch provides device memory (tensors) and streams; it is
imported before the library is loaded so that both share one HIP runtime (both carry the soname
libamdhip64.so.7, and the first one loaded is reused).

There is no fallback: if the library is missing or a call fails, an exception is raised.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtrivance.so")

LATENCY_OPT, BANDWIDTH_OPT, BRUCK_REF = 0, 1, 2
F32, I32 = 0, 1
ROUTE_SCHEDULED, ROUTE_SHORTEST = 0, 1
PHASE_LATENCY, PHASE_REDUCE_SCATTER, PHASE_ALLGATHER = 0, 1, 2
MAX_DIMS = 8

_VARIANTS = {"L": LATENCY_OPT, "B": BANDWIDTH_OPT, "BRUCK": BRUCK_REF}
PLACE_BY_SCHEDULE = 1  # TRIVANCE_PLACE_BY_SCHEDULE
_PLACEMENTS = {"natural": 0, "schedule": PLACE_BY_SCHEDULE}
_ROUTING = {"scheduled": ROUTE_SCHEDULED, "shortest": ROUTE_SHORTEST}


class TrivanceError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what} failed: {_lib().trivance_strerror(status).decode()} ({status})")


class CostResult(ctypes.Structure):
    _fields_ = [("total", ctypes.c_double), ("latency", ctypes.c_double),
                ("transmission", ctypes.c_double), ("theta", ctypes.c_double),
                ("passes", ctypes.c_int)]


class Topology(ctypes.Structure):
    _fields_ = [("ndims", ctypes.c_int), ("dims", ctypes.c_int * MAX_DIMS),
                ("routing", ctypes.c_int)]


_LIB = None


def _lib():
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                           "(python -m paper_2602_17254_amd._build)")
    import torch  # noqa: F401  -- load torch's HIP runtime first (see module docstring)

    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    i64 = ctypes.c_int64
    sig = {
        "trivance_plan": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(ctypes.c_int), ctypes.c_int,
                                         ctypes.c_int, ctypes.POINTER(P)]),
        "trivance_plan_ex": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(ctypes.c_int), ctypes.c_int,
                                            ctypes.c_int, ctypes.c_uint, ctypes.POINTER(P)]),
        "trivance_plan_destroy": (None, [P]),
        "trivance_plan_num_steps": (ctypes.c_int, [P]),
        "trivance_plan_num_passes": (ctypes.c_int, [P]),
        "trivance_plan_step": (ctypes.c_int, [P, ctypes.c_int, ctypes.c_int] +
                               [ctypes.POINTER(ctypes.c_int)] * 3),
        "trivance_plan_step_index": (ctypes.c_int, [P, ctypes.c_int]),
        "trivance_plan_with_dispatch_limit": (ctypes.c_int, [P, i64, ctypes.POINTER(P)]),
        "trivance_block_range": (ctypes.c_int, [P, i64, ctypes.c_int, ctypes.c_int,
                                                ctypes.POINTER(i64), ctypes.POINTER(i64)]),
        "trivance_algorithmic_bytes": (i64, [P, i64, ctypes.c_int]),
        "trivance_pass_bytes": (i64, [P, i64, ctypes.c_int, ctypes.c_int]),
        "trivance_allreduce_emulated": (ctypes.c_int, [P, ctypes.c_int, i64, ctypes.c_int, P, P]),
        "trivance_allreduce_emulated_steps": (ctypes.c_int, [P, ctypes.c_int, i64, ctypes.c_int,
                                                             P, P, ctypes.c_int, ctypes.c_int]),
        "trivance_workspace_bytes": (i64, [P, i64, ctypes.c_int]),
        "trivance_allreduce_emulated_ws": (ctypes.c_int, [P, ctypes.c_int, i64, ctypes.c_int, P, P,
                                                          i64, P]),
        "trivance_allreduce_emulated_steps_ws": (ctypes.c_int, [P, ctypes.c_int, i64, ctypes.c_int,
                                                                P, P, i64, P, ctypes.c_int,
                                                                ctypes.c_int]),
        "trivance_congestion": (i64, [P, ctypes.POINTER(Topology), ctypes.POINTER(i64), i64]),
        "trivance_congestion_device": (ctypes.c_int, [P, ctypes.POINTER(Topology), P, i64, P]),
        "trivance_congestion_noalloc": (i64, [P, ctypes.POINTER(Topology), ctypes.POINTER(i64), i64]),
        "trivance_fill_hash_uniform": (ctypes.c_int, [P, ctypes.c_int, i64, ctypes.c_uint64, P]),
        "trivance_copy_device": (ctypes.c_int, [P, P, i64, P]),
        "trivance_cost_model": (ctypes.c_int, [P, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                               ctypes.POINTER(ctypes.c_double), ctypes.c_int,
                                               ctypes.POINTER(CostResult)]),
        "trivance_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def exported_symbols() -> list:
    """Names the binding resolves (all of include/trivance.h)."""
    lib = ctypes.CDLL(LIB_PATH)
    names = ["trivance_plan", "trivance_plan_ex", "trivance_plan_destroy", "trivance_plan_num_steps",
             "trivance_plan_num_passes", "trivance_plan_step", "trivance_plan_step_index",
             "trivance_plan_with_dispatch_limit", "trivance_block_range",
             "trivance_algorithmic_bytes", "trivance_pass_bytes", "trivance_allreduce_emulated",
             "trivance_allreduce_emulated_steps", "trivance_workspace_bytes",
             "trivance_allreduce_emulated_ws", "trivance_allreduce_emulated_steps_ws",
             "trivance_congestion",
             "trivance_congestion_device", "trivance_congestion_noalloc", "trivance_fill_hash_uniform",
             "trivance_copy_device", "trivance_cost_model", "trivance_strerror"]
    return [n for n in names if hasattr(lib, n)]


def _check(rc: int, what: str) -> int:
    if rc < 0:
        raise TrivanceError(int(rc), what)
    return rc


class Plan:
    """Owns a trivance_plan_t handle."""

    def __init__(self, handle, dims, variant, placement="natural"):
        self._h = handle
        self.dims = tuple(dims)
        self.variant = variant
        self.placement = placement
        self.n = int(np.prod(self.dims))
        self.D = len(self.dims)

    @property
    def handle(self):
        return self._h

    @property
    def num_steps(self) -> int:
        return _check(_lib().trivance_plan_num_steps(self._h), "trivance_plan_num_steps")

    @property
    def num_passes(self) -> int:
        return _check(_lib().trivance_plan_num_passes(self._h), "trivance_plan_num_passes")

    def __del__(self):
        if getattr(self, "_h", None) and _LIB is not None:
            _LIB.trivance_plan_destroy(self._h)
            self._h = None


def trivance_plan(dims, variant="L", placement="natural") -> Plan:
    """Build a plan for a ring (dims=(n,)) or torus; variant 'L', 'B' or 'BRUCK'; placement
    'natural' (block j at the j-th granule range) or 'schedule' (TRIVANCE_PLACE_BY_SCHEDULE)."""
    dims = tuple(int(d) for d in dims)
    arr = (ctypes.c_int * len(dims))(*dims)
    h = ctypes.c_void_p()
    n = int(np.prod(dims)) if dims else 0
    _check(_lib().trivance_plan_ex(n, arr, len(dims), _VARIANTS[variant], _PLACEMENTS[placement],
                                   ctypes.byref(h)), "trivance_plan_ex")
    return Plan(h, dims, variant, placement)


def trivance_plan_step(plan: Plan, pass_index: int, collective: int = 0) -> tuple:
    """(phase, dim, distance) of one pass for one collective."""
    out = [ctypes.c_int() for _ in range(3)]
    _check(_lib().trivance_plan_step(plan.handle, pass_index, collective,
                                     *[ctypes.byref(o) for o in out]), "trivance_plan_step")
    return tuple(o.value for o in out)


def trivance_plan_step_index(plan: Plan, pass_index: int) -> int:
    """Global step index t that a pass materialises (all-gather passes run t = S-1 .. 0)."""
    return _check(_lib().trivance_plan_step_index(plan.handle, pass_index),
                  "trivance_plan_step_index")


def trivance_plan_with_dispatch_limit(plan: Plan, work_items: int) -> Plan:
    """A new plan equal to `plan` whose launches are issued as dispatches of at most `work_items`
    work-items (1024 .. 2^31); `plan` itself is unchanged."""
    h = ctypes.c_void_p()
    _check(_lib().trivance_plan_with_dispatch_limit(plan.handle, int(work_items), ctypes.byref(h)),
           "trivance_plan_with_dispatch_limit")
    return Plan(h, plan.dims, plan.variant, plan.placement)


def trivance_block_range(plan: Plan, elems: int, collective: int, block: int) -> tuple:
    b, e = ctypes.c_int64(), ctypes.c_int64()
    _check(_lib().trivance_block_range(plan.handle, elems, collective, block, ctypes.byref(b),
                                       ctypes.byref(e)), "trivance_block_range")
    return b.value, e.value


def trivance_algorithmic_bytes(plan: Plan, elems: int, dtype: int = F32) -> int:
    return _check(_lib().trivance_algorithmic_bytes(plan.handle, elems, dtype),
                  "trivance_algorithmic_bytes")


def trivance_pass_bytes(plan: Plan, elems: int, pass_index: int, dtype: int = F32) -> int:
    return _check(_lib().trivance_pass_bytes(plan.handle, elems, dtype, pass_index),
                  "trivance_pass_bytes")


def _stream_ptr(stream):
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _buffer_args(buffers, plan: Plan):
    import torch

    if not isinstance(buffers, torch.Tensor) or not buffers.is_cuda:
        raise TypeError("buffers must be a CUDA (HIP) torch tensor")
    if buffers.dim() != 2 or buffers.shape[0] != plan.n or not buffers.is_contiguous():
        raise ValueError(f"buffers must be a contiguous [{plan.n}, elems] tensor")
    if buffers.dtype == torch.float32:
        dt = F32
    elif buffers.dtype == torch.int32:
        dt = I32
    else:
        raise TypeError("buffers must be float32 or int32")
    return ctypes.c_void_p(buffers.data_ptr()), plan.n, buffers.shape[1], dt


def trivance_allreduce_emulated(buffers, plan: Plan, stream=None) -> None:
    """In-place emulated AllReduce over the rows of `buffers` (enqueued on `stream`)."""
    ptr, n, E, dt = _buffer_args(buffers, plan)
    _check(_lib().trivance_allreduce_emulated(ptr, n, E, dt, plan.handle, _stream_ptr(stream)),
           "trivance_allreduce_emulated")


def trivance_allreduce_emulated_steps(buffers, plan: Plan, pass_begin: int, pass_end: int,
                                      stream=None) -> None:
    ptr, n, E, dt = _buffer_args(buffers, plan)
    _check(_lib().trivance_allreduce_emulated_steps(ptr, n, E, dt, plan.handle,
                                                    _stream_ptr(stream), pass_begin, pass_end),
           "trivance_allreduce_emulated_steps")


def trivance_workspace_bytes(plan: Plan, elems: int, dtype: int = F32) -> int:
    return _check(_lib().trivance_workspace_bytes(plan.handle, elems, dtype),
                  "trivance_workspace_bytes")


def _workspace_args(workspace):
    import torch

    if workspace is None:
        return ctypes.c_void_p(0), 0
    if not isinstance(workspace, torch.Tensor) or not workspace.is_cuda or \
            not workspace.is_contiguous():
        raise TypeError("workspace must be a contiguous CUDA tensor")
    return ctypes.c_void_p(workspace.data_ptr()), workspace.numel() * workspace.element_size()


def trivance_allreduce_emulated_ws(buffers, plan: Plan, workspace, stream=None) -> None:
    """In-place emulated AllReduce with a caller-owned device workspace (any contiguous CUDA tensor
    of at least trivance_workspace_bytes bytes)."""
    ptr, n, E, dt = _buffer_args(buffers, plan)
    wp, wb = _workspace_args(workspace)
    _check(_lib().trivance_allreduce_emulated_ws(ptr, n, E, dt, plan.handle, wp, wb,
                                                 _stream_ptr(stream)),
           "trivance_allreduce_emulated_ws")


def trivance_allreduce_emulated_steps_ws(buffers, plan: Plan, workspace, pass_begin: int,
                                         pass_end: int, stream=None) -> None:
    ptr, n, E, dt = _buffer_args(buffers, plan)
    wp, wb = _workspace_args(workspace)
    _check(_lib().trivance_allreduce_emulated_steps_ws(ptr, n, E, dt, plan.handle, wp, wb,
                                                       _stream_ptr(stream), pass_begin, pass_end),
           "trivance_allreduce_emulated_steps_ws")


def _topology(plan: Plan, routing: str) -> Topology:
    t = Topology()
    t.ndims = plan.D
    for i, d in enumerate(plan.dims):
        t.dims[i] = d
    t.routing = _ROUTING[routing]
    return t


def trivance_congestion(plan: Plan, routing: str = "scheduled") -> np.ndarray:
    """int64 loads[pass][rank][port] computed on the GPU (synchronous)."""
    lib = _lib()
    topo = _topology(plan, routing)
    need = _check(lib.trivance_congestion(plan.handle, ctypes.byref(topo), None, 0),
                  "trivance_congestion")
    out = np.zeros(need, dtype=np.int64)
    _check(lib.trivance_congestion(plan.handle, ctypes.byref(topo),
                                   out.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), need),
           "trivance_congestion")
    return out.reshape(plan.num_passes, plan.n, 2 * plan.D)


def trivance_congestion_noalloc(plan: Plan, routing: str = "scheduled") -> np.ndarray:
    """trivance_congestion computed in the library's fixed device scratch (no device allocation;
    at most 2^20 entries)."""
    lib = _lib()
    topo = _topology(plan, routing)
    need = _check(lib.trivance_congestion_noalloc(plan.handle, ctypes.byref(topo), None, 0),
                  "trivance_congestion_noalloc")
    out = np.zeros(need, dtype=np.int64)
    _check(lib.trivance_congestion_noalloc(plan.handle, ctypes.byref(topo),
                                           out.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), need),
           "trivance_congestion_noalloc")
    return out.reshape(plan.num_passes, plan.n, 2 * plan.D)


def trivance_congestion_device(plan: Plan, out, routing: str = "scheduled", stream=None) -> None:
    """Same counts written into a caller-owned int64 CUDA tensor (asynchronous)."""
    import torch

    if not isinstance(out, torch.Tensor) or not out.is_cuda or out.dtype != torch.int64 \
            or not out.is_contiguous():
        raise TypeError("out must be a contiguous int64 CUDA tensor")
    topo = _topology(plan, routing)
    _check(_lib().trivance_congestion_device(plan.handle, ctypes.byref(topo),
                                             ctypes.c_void_p(out.data_ptr()), out.numel(),
                                             _stream_ptr(stream)), "trivance_congestion_device")


def trivance_fill_hash_uniform(buffers, seed: int, stream=None) -> None:
    """Fill a float32 [n, elems] CUDA tensor with the counter-based U(-1, 1) inputs."""
    import torch

    if not isinstance(buffers, torch.Tensor) or not buffers.is_cuda or buffers.dtype != torch.float32 \
            or buffers.dim() != 2 or not buffers.is_contiguous():
        raise TypeError("buffers must be a contiguous float32 [n, elems] CUDA tensor")
    _check(_lib().trivance_fill_hash_uniform(ctypes.c_void_p(buffers.data_ptr()),
                                             buffers.shape[0], buffers.shape[1], seed,
                                             _stream_ptr(stream)), "trivance_fill_hash_uniform")


def trivance_copy_device(dst, src, stream=None) -> None:
    """Benchmark helper: copy the contiguous CUDA tensor `src` into `dst` (the same number of
    bytes, a multiple of 16) with the library's streaming copy kernel."""
    import torch

    for name, t in (("dst", dst), ("src", src)):
        if not isinstance(t, torch.Tensor) or not t.is_cuda or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous CUDA tensor")
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nbytes:
        raise ValueError("dst and src must hold the same number of bytes")
    _check(_lib().trivance_copy_device(ctypes.c_void_p(dst.data_ptr()),
                                       ctypes.c_void_p(src.data_ptr()), nbytes,
                                       _stream_ptr(stream)), "trivance_copy_device")


def trivance_cost_model(plan: Plan, bytes_per_rank: float, alpha: float = 0.0,
                        beta: float = 0.0) -> dict:
    """The Sec. 2.1 cost model of the plan for an AllReduce of `bytes_per_rank` bytes per rank:
    total, latency and transmission times, theta, passes, and the busiest link's bytes per
    pass."""
    P = plan.num_passes
    peaks = (ctypes.c_double * max(P, 1))()
    res = CostResult()
    _check(_lib().trivance_cost_model(plan.handle, float(bytes_per_rank), float(alpha), float(beta),
                                      peaks, max(P, 1), ctypes.byref(res)), "trivance_cost_model")
    return {"total": res.total, "latency": res.latency, "transmission": res.transmission,
            "theta": res.theta, "passes": res.passes, "pass_link_bytes": list(peaks)[:P]}
