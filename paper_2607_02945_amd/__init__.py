"""MI355X (gfx950) grouped execution of many independent small operators.

The runtime effect of the horizontal group fusion and vertical split-concat
rewrites of "Optimus" (KDD '26): one kernel launch per operator type for a
group of independent Linear / LayerNorm / pointwise operators, and a fused
split -> per-piece op -> concat that makes no intermediate copies.

The work runs in liboptimus.so (hand-written HIP kernels, C ABI in
include/optimus.h); ``binding`` marshals torch tensors into its descriptors.
"""
from .binding import (  # noqa: F401
    OptimusError,
    Plan,
    optimus_grouped_layernorm,
    optimus_grouped_linear,
    optimus_grouped_pointwise,
    optimus_last_error,
    optimus_plan_layernorm,
    optimus_plan_linear,
    optimus_plan_pointwise,
    optimus_plan_split_op_cat,
    optimus_split_op_cat,
    optimus_validate_layernorm,
    optimus_validate_linear,
    optimus_validate_pointwise,
    optimus_validate_split_op_cat,
    optimus_version,
)
