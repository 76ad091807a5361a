"""MI355X (gfx950) hot path of the Mixture Compressor MoE method.

Thin Python binding of ``libmcmoe.so`` (C-ABI in ``include/mc_moe.h``): every
step runs in the HIP kernels; this module only marshals torch device tensors
into the C descriptors and passes the current stream.  It raises if the
library is not built -- there is no fallback.
"""
from ._binding import (  # noqa: F401
    MCError,
    QUANT_RTN,
    QUANT_SIGN,
    PackedLayer,
    Routing,
    codes_export,
    dequant_export,
    forward_workspace,
    gptq_factor,
    gptq_hessian,
    gptq_quantize,
    gptq_workspace,
    importance_workspace,
    lib_path,
    load,
    moe_forward,
    moe_forward_noalloc,
    odp_threshold,
    pack,
    pack_sizes,
    pmq_allocate,
    pmq_error_workspace,
    pmq_expert_error,
    pmq_significance,
    route_and_prune,
    route_forward,
    router_logits,
    stack_forward,
    stack_workspace,
    timing_enable,
    timing_read,
    token_importance,
)
