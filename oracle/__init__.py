"""CPU oracle for the LLEP expert-layer hot path.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke entry point and the CPU
baseline leg of the benchmark may import or call anything in this package.
The product path (the HIP library and its binding) never does, and shares no
code, table or helper with it.

Everything here is plain and slow on purpose: Python integers for the plan,
plain counting for the permutation, float64 numpy arithmetic for the expert
outputs. Each function cites the passage of the paper it follows.
"""

from .backward import (  # noqa: F401
    combine_backward,
    moe_backward,
    plan_backward,
    silu_grad,
    swiglu_ffn_backward,
)
from .llep import (  # noqa: F401
    DeviceLedger,
    PlanResult,
    bypass_to_standard_ep,
    capacity_from_alpha,
    combine,
    expert_loads,
    least_loaded_assignment,
    m_local,
    min_max_load_exhaustive,
    moe_output,
    pair_ranks,
    permute,
    plan,
    plan_tables,
    silu,
    spill_to_least_loaded,
    standard_ep_assignment,
    swiglu_ffn,
)
