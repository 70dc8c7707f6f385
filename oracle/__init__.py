"""Plain fp64 CPU oracle of the SPLA decode step (test infrastructure only).

This package is test infrastructure. Only the test-suite, the smoke check and
the CPU-baseline leg of the benchmark may import it; the product path (the HIP
library and its Python binding) never does, and this package imports nothing
from the product.

Paper: "SPLA: Block Sparse Plus Linear Attention for Long Context Modeling"
(arXiv 2601.22379), Sections 2 and 3.
"""

from .spla_oracle import (  # noqa: F401
    SplaParams,
    KVState,
    DecodeResult,
    block_ranges,
    block_stats,
    window_ranges,
    window_stats,
    pool_windows_to_blocks,
    feature_map,
    global_state,
    log_block_mass,
    group_block_scores,
    forced_blocks,
    select_blocks,
    selected_token_indices,
    exact_sparse_attention,
    nothing_unselected,
    residual_linear_attention,
    combine,
    build_state,
    decode_kv_head,
    decode_from_state,
    decode_sequence,
    append_state,
    cutoff_score,
    prefill_kv_head,
)
