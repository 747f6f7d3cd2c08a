"""Plain fp64 CPU oracle of the MoE layer forward and backward.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only the tests, the package's smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the HIP path.
"""
from .moe_oracle import (  # noqa: F401
    RouterSpec,
    spec_from_config,
    router_logits,
    route,
    sort_maps,
    permute_rows,
    glu,
    expert_forward,
    expert_backward,
    layer_forward,
    layer_backward,
    router_backward,
    threshold_backward,
    combine,
    combine_backward,
    unpermute,
    token_forward_backward,
    expert_weight_grads_at,
    router_probs,
    aux_loss,
    aux_loss_backward,
    ZeroComputeSpec,
    zc_kind,
    zc_aux_weights,
    zc_const_alpha,
    zc_forward,
    zc_backward,
    e4m3_values,
    e4m3_round,
    quantize_rows,
    quantize_cols,
    fp8_expert_backward,
    fp8_expert_forward,
)
