"""sdattn for MI355X: SD1.4 UNet attention as hand-written HIP kernels for gfx950.

The compute lives in ``libsdattn.so`` (C ABI declared in ``include/sdattn.h``).
This package is a thin binding: it marshals torch tensors' device pointers and
the current HIP stream into that library and raises on a nonzero status.  The
library is loaded on first use; if it is missing the call raises instead of
falling back to anything else.
"""
from .binding import (  # noqa: F401
    SdattnError, forward, forward_ex, softmax_rows, logits, softmax_pv, linear,
    attention_block_workspace, attention_block, attention_block_static, project_kv, attention_block_kv, group_norm, geglu,
    winograd_weights, conv3x3_workspace, conv3x3,
    library_path,
    load_library,
    LAYOUT_ROWS, LAYOUT_HEADS,
    STATUS_OK, STATUS_INVALID_ARG, STATUS_UNSUPPORTED, STATUS_MISALIGNED, STATUS_HIP, STATUS_SCRATCH,
    DTYPE_F16, DTYPE_BF16, DTYPE_F32,
)
