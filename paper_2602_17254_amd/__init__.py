"""MI355X-native emulated Trivance AllReduce (arXiv 2602.17254).

The native library (libtrivance.so, C ABI in include/trivance.h) holds the schedule generator and
the gfx950 kernels; `binding` marshals arguments to it; `inputs` produces seeded synthetic inputs.
"""

from .binding import (  # noqa: F401
    BANDWIDTH_OPT, BRUCK_REF, F32, I32, LATENCY_OPT, Plan, TrivanceError, trivance_algorithmic_bytes,
    trivance_allreduce_emulated, trivance_allreduce_emulated_steps, trivance_allreduce_emulated_steps_ws,
    trivance_allreduce_emulated_ws, trivance_block_range, trivance_workspace_bytes,
    trivance_congestion, trivance_congestion_device, trivance_copy_device, trivance_cost_model,
    trivance_fill_hash_uniform,
    trivance_pass_bytes, trivance_plan, trivance_plan_step, trivance_plan_step_index,
    trivance_plan_with_dispatch_limit)
