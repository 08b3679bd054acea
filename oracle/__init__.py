"""fp64 CPU oracle for the fused draft-verify step (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package; the library never does.
"""
from .recguide_oracle import (  # noqa: F401
    ar_mask,
    bf16_bits_to_f64,
    diffusion_mask,
    entropy_row,
    first_argmax,
    fused_step_mask,
    gather_request_kv,
    oracle_accept,
    oracle_attention,
    oracle_confidence,
    softmax_attention,
    softmax_row,
)
from .branches import (  # noqa: F401
    branch_step_mask,
    oracle_branch_attention,
    oracle_match_branches,
    oracle_plan_branches,
    request_branches,
)
from .blocksize import (  # noqa: F401
    oracle_block_state,
    oracle_bucket,
    oracle_plan_block_sizes,
    oracle_route,
    oracle_utilities,
    s_bin,
)
