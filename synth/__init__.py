"""Seeded synthetic workloads for the HSA active-token layer step.

This package only draws inputs (random latents, weights, budgets, caches) and
describes the workload shapes. It holds none of the method's arithmetic: no
active-set rule, no projection, no attention, no Euler update. Both the CPU
oracle and the GPU path consume what it produces.
"""

from .workloads import (  # noqa: F401
    PRESETS,
    WORKLOADS,
    Workload,
    assign_budgets,
    bf16_tensor,
    draw_block,
    draw_cache,
    draw_euler_state,
    draw_stack,
    draw_stack_state,
    group_sizes,
    linear_sigmas,
    random_budgets,
    to_bf16_values,
)
