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
    LossCall,
    lambda_from_logodds,
    library_path,
    load_library,
    loss_bwd,
    loss_fwd,
    read_stats,
    status_string,
    weights,
    workspace_bytes,
)

__all__ = [
    "CisError", "CIS_BF16", "CIS_F32", "LossCall", "lambda_from_logodds", "library_path", "load_library",
    "loss_bwd", "loss_fwd", "read_stats", "status_string", "weights", "workspace_bytes",
]
