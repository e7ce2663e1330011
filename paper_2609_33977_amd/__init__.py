"""MI355X-native group-masked linear layer of GroupMask (gfx950 HIP kernels behind a C ABI).

Importing this package loads libgroupmask.so and fails if it has not been built.
"""
from ._lib import (  # noqa: F401
    GM_OK, GM_ERR_NULL, GM_ERR_SHAPE, GM_ERR_VALUE, GM_ERR_ALIGN, GM_ERR_WORKSPACE, GM_ERR_DEVICE,
    GM_OP_FWD, GM_OP_BWD, EXPORTS, LIB, LIB_PATH, GroupMaskError, status_string,
    gm_abi_version, gm_gate, gm_gate_bwd, gm_budget_loss, gm_gate_bwd_budget, gm_workspace_size,
    gm_masked_linear_fwd, gm_masked_linear_bwd, gm_masked_linear_bwd_noalloc, GM_NOALLOC_SCRATCH_BYTES,
    gm_pack_rows, gm_packed_linear_fwd,
    gm_distill_workspace_size, gm_distill_fwd, gm_distill_bwd,
    gm_hyper_workspace_size, gm_hyper_fwd, gm_hyper_bwd, gm_adamw,
)
