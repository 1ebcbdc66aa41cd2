"""MI355X (gfx950) calibrated-importance-sampling (CIS) token loss, forward and backward.

Thin Python binding over libcis.so (see include/cis.h): it checks tensor arguments, allocates
outputs and the workspace with torch, and passes device pointers plus torch's current HIP
stream to the C ABI. Every step of the computation runs in the library's HIP kernels; there is
no fallback path.
"""

from ._binding import (  # noqa: F401
    CisError,
    CIS_BF16,
    CIS_F32,
    LMHEAD_CHUNK,
    LossCall,
    NOALLOC_MAX_T,
    OP_CIS,
    OP_EXACT,
    OP_ICEPOP,
    OP_KPOP,
    OP_NONE,
    OP_QFIXED,
    OP_SEQ_MIS,
    OP_SEQ_TIS,
    OP_TIS,
    OP_TWO_SIDED,
    Params,
    SEQ_OPS,
    lambda_from_logodds,
    library_path,
    lmhead_loss_bwd,
    lmhead_loss_fwd,
    lmhead_workspace_bytes,
    load_library,
    loss_bwd,
    loss_bwd_ex,
    loss_bwd_noalloc,
    loss_fwd,
    loss_fwd_ex,
    params,
    read_stats,
    status_string,
    weights,
    weights_ex,
    workspace_bytes,
    workspace_bytes_ex,
)

__all__ = [
    "CisError", "CIS_BF16", "CIS_F32", "LMHEAD_CHUNK", "LossCall", "NOALLOC_MAX_T", "OP_CIS", "OP_EXACT", "OP_ICEPOP", "OP_KPOP",
    "OP_NONE", "OP_QFIXED", "OP_SEQ_MIS", "OP_SEQ_TIS", "OP_TIS", "OP_TWO_SIDED", "Params",
    "SEQ_OPS", "lambda_from_logodds", "library_path", "lmhead_loss_bwd", "lmhead_loss_fwd",
    "lmhead_workspace_bytes", "load_library", "loss_bwd", "loss_bwd_ex", "loss_bwd_noalloc",
    "loss_fwd", "loss_fwd_ex", "params", "read_stats", "status_string", "weights", "weights_ex",
    "workspace_bytes", "workspace_bytes_ex",
]
