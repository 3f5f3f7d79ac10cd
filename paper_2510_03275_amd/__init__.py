"""SDQ-LLM hot path on MI355X: Sigma-Delta weight encoder and addition-only
linear layer as hand-written HIP kernels for gfx950 behind a C ABI
(include/sdq.h).  This package is the thin Python binding of that library."""
from .binding import (  # noqa: F401
    Encoded, SdqError, lib, linear, quantize, sdq_codes_bytes, sdq_compression_ratio, sdq_layout,
    sdq_layout_init, sdq_layout_set_hadamard, sdq_layout_set_packing, sdq_linear, sdq_expand_activations,
    sdq_linear_expanded, sdq_linear_workspace_bytes, sdq_moments_workspace_bytes,
    sdq_multiosr, sdq_prepare, sdq_prepare_layout, sdq_quantize, sdq_quantize_check,
    sdq_quantize_workspace_bytes, sdq_release_tables, sdq_unpack_codes, sdq_upsample_table,
    sdq_version, sdq_weight_moments, sdq_hessian_accumulate, sdq_hessian_factor,
    sdq_hessian_factor_workspace_bytes, sdq_hessian_check, sdq_quantize_compensated,
    sdq_quantize_compensated_workspace_bytes, hessian_factor, quantize_compensated,
    SDQ_F16, SDQ_BF16, SDQ_F32, SDQ_HAD_NONE, SDQ_HAD_SYLVESTER, SDQ_HAD_SIGNED, SDQ_PACK_FIELDS, SDQ_PACK_BASE3,
    SDQ_COMP_GPTQ, SDQ_COMP_JOINT, SDQ_NOALLOC_SCRATCH_BYTES, sdq_linear_noalloc,
    LinearGroup, sdq_linear_group, sdq_linear_group_workspace_bytes, sdq_linear_group_expanded,
)
