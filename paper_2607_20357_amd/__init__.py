"""Budget-adapted MLLM prefill (SmartVL inference path) on MI355X.

The computation lives in libsvl.so (hand-written HIP kernels for gfx950
behind a C ABI, see include/svl.h); `binding` marshals torch tensors and
numpy arrays into its calls.
"""
from .binding import (  # noqa: F401
    CONTROLLER_FIELDS, KCLASS, SVL_BF16, SVL_COMPUTE_BF16, SVL_COMPUTE_F16, SVL_F32, Controller,
    LayerTable, SvlError, alloc_controlled_workspace, alloc_decode_workspace, alloc_kv_cache,
    alloc_workspace, layer_weights, load_library, make_config, svl_abi_version,
    svl_budget_loss, svl_budget_loss_params, svl_budget_project, svl_controlled_workspace_bytes, svl_count_flops, svl_count_positive,
    svl_decode_step, svl_decode_step_noalloc, svl_kv_cache_bytes, svl_layer_forward, svl_prefill, svl_prefill_cache,
    svl_prefill_controlled, svl_select_tokens, svl_timing_enable, svl_timing_read,
    svl_workspace_bytes, alloc_train_workspace, svl_train_params, svl_train_step,
    SVL_STATUS_NONFINITE, svl_workspace_status,
    svl_train_workspace_bytes,
)
