"""fp64 CPU oracle of the SAF3R hot path (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package; the product path never does.
"""
from .saf3r_oracle import *  # noqa: F401,F403
from .saf3r_oracle import (  # noqa: F401
    ANCHOR,
    DENSE,
    FRAME_LOCAL,
    GLOBAL_PROBE,
    STRIDE,
    TOPK,
    anchor_row,
    COSINE_TOPK,
    attend_block,
    attend_head,
    attend_stride,
    attention_flops,
    baseline_stride,
    attend_tokens,
    block_range,
    block_frame,
    block_scores,
    cosine_block_features,
    cosine_topk_row,
    dense_attention,
    frame_local_row,
    global_probe_row,
    kept_fraction,
    nmse,
    num_blocks,
    pool_blocks,
    progressive_substitution,
    run_layer,
    select_head,
    stride_keys,
    to_f64,
    topk_row,
)
