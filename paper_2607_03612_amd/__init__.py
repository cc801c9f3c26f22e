"""SAF3R block-sparse global attention for AMD Instinct MI355X (gfx950).

The compute path is the HIP library ``libsaf3r.so`` (C ABI in
``include/saf3r.h``); ``binding`` marshals torch device tensors into it.
"""
from . import binding  # noqa: F401
from .binding import (  # noqa: F401
    ANCHOR,
    BF16,
    COSINE_TOPK,
    DENSE,
    F32,
    FRAME_LOCAL,
    GLOBAL_PROBE,
    TOPK,
    Saf3rError,
    attention_workspace_bytes,
    cosine_select,
    cosine_workspace_bytes,
    estimate_blocks,
    index_capacity,
    load,
    nmse,
    nmse_noalloc,
    nmse_workspace_bytes,
    num_blocks,
    run_layer,
    select_blocks,
    select_workspace_bytes,
    SKIP,
    sparse_attention,
    STRIDE,
    validate_index,
)
