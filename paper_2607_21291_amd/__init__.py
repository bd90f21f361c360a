"""MI355X (gfx950) depth-sparse Transformer layer forward (AdaDSF), with the
router-score pathway of its training side (score gating and router backward).

The compute lives in the HIP library ``libadadsf.so`` (C ABI in
``include/adadsf.h``); this package is its thin Python binding.
"""
from ._binding import (  # noqa: F401
    BF16, BLOCK_NEOX_PARALLEL, BLOCK_QWEN_SEQ, EXPORTS, F32, FLAG_DENSE, FLAG_GATE, KINDS, DeviceLayer, DsfError,
    LayerDesc, LayerWeights, align_hidden, align_stack_forward, align_stack_workspace_size, align_workspace_size,
    decode_step, decode_workspace_size, stack_prefill, decode_step_static, decode_static_scratch_bytes,
    attention_forward, kl_align, gate_score_grad, gather_rows, k_from_retention, last_error, lib,
    make_desc, retention_from_similarity, router_backward, router_backward_workspace_size, router_score, scatter_residual, sim_finalize, sim_stats, sim_workspace_size,
    sparse_block_forward, stack_forward, timing_enable, timing_read, topk_select, version, workspace_size,
    workspace_status, WS_STATUS_SK_TIMEOUT, backward_workspace_size, sparse_block_backward, GRAD_FIELDS,
    LayerGrads,
)
