"""CPU oracle for the HSA active-token layer step (test infrastructure only).

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
import this package; the product path never does. It shares no code with the
HIP library.
"""

from .hsa_oracle import (  # noqa: F401
    active_set,
    attention,
    attention_output,
    cached_euler,
    check_budgets,
    euler_delta,
    layer_step,
    mean_steps,
    project,
    qkv_cache_update,
    round_bf16,
    round_f32,
    round_to,
    trajectory,
    window_margin,
)
from .stack_oracle import (  # noqa: F401
    SELECT_L1REL,
    SELECT_NORM,
    ROPE_THETA,
    apply_rope,
    assign_by_key,
    assign_groups,
    boundary_gaps,
    check_group_sizes,
    gather_latent,
    gelu_tanh,
    initial_state,
    l1_rel,
    linear,
    refresh_period,
    reorder_plan,
    rms_normalize,
    rope_angles,
    rope_bands,
    RMS_EPS,
    stack_forward,
    stack_iteration,
    stack_trajectory,
    token_ranks,
    velocity_keys,
)
