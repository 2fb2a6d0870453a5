"""MI355X (gfx950) HIP implementation of the MoE-layer hot path of FlowMoE
(arXiv 2510.00207): gating with top-k, capacity-bounded dispatch into the
expert-major send layout, grouped-GEMM expert FFNs, combine, their backward,
and the R-chunk two-stream schedule.

The compute lives in libflowmoe.so (C ABI in include/flowmoe.h); this package
is its ctypes binding (`_lib`, names identical to the C entry points) plus a
buffer helper (`layer.MoELayer`).
"""
from ._lib import (  # noqa: F401
    BF16, F32, GATE_FULL, GATE_RENORM, GELU, PACKED, PADDED, SWIGLU, WS_DISPATCH, WS_FFN_BWD,
    WS_GATE_BWD, WS_LAYER_BWD,
    FlowMoEError, LayerBufs, Shape, flowmoe_capacity, flowmoe_combine, flowmoe_combine_bwd,
    flowmoe_dispatch, flowmoe_dispatch_bwd, flowmoe_expert_ffn, flowmoe_expert_ffn_bwd,
    flowmoe_gate_topk, flowmoe_gate_topk_bwd, flowmoe_last_error, flowmoe_layer_bwd,
    flowmoe_layer_fwd, flowmoe_route, flowmoe_rows_capacity, flowmoe_version,
    flowmoe_workspace_bytes, layer_bufs, load, make_shape,
)
