"""FrameFT adapter hot path on MI355X (gfx950): HIP kernels behind a C ABI.

The compute lives in ``libframeft.so`` (built from ``csrc/``); the Python
names below only marshal arguments to it.  Importing this package does not
load the library; the first call does, and fails loudly if it is missing.
"""
from .binding import (  # noqa: F401
    Frame, Plan, FrameFTError, framegen, tff_host, plan_create, adapter_fwd,
    adapter_bwd, merge_delta, adapter_fwd_batched, adapter_bwd_batched, coef_to_plan,
    coef_to_user, adamw_step, adamw_step_batched, lr_linear_warmup, PlanGroup, plan_group, adapter_fwd_group,
    adapter_bwd_group, library_path,
)
