"""CPU oracle of the MoE-layer forward pass (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package. The GPU path never does.
"""

from .oracle import (  # noqa: F401
    BIAS_SIGN,
    BIAS_ZSCORE,
    bias_update,
    build_oracle,
    combine,
    expert_backward,
    expert_rows,
    gelu,
    gelu_grad,
    grouped_backward,
    layer,
    logits,
    num_threads,
    permute,
    round_bf16,
    route,
    scores,
    sigmoid,
    silu,
    silu_grad,
    topk_from_scores,
)
