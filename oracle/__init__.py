"""Plain CPU reference of FlexPrefill (arXiv 2502.20766) -- TEST INFRASTRUCTURE ONLY.

This package is the oracle that the device path is checked against.  Only the test
suite, the smoke check and the benchmark's CPU-baseline leg may import it; the
product path (the HIP library and its Python binding) never does, and shares no
code with it.

Everything is float64 numpy, one (sequence, query head) at a time, written as the
paper's definitions and algorithm steps in the paper's order, with no blocking or
fusion beyond what a definition states.  Readings of points the paper leaves open
are marked "Reading:" where they are taken.
"""
from .flexprefill import (  # noqa: F401
    PATTERN_QA,
    PATTERN_VS,
    PATTERN_DENSE,
    representative_queries,
    representative_attention,
    vertical_slash_scores,
    true_block_distribution,
    estimated_block_distribution,
    js_distance,
    sparse_pattern_search,
    cumulative_select,
    vertical_slash_index,
    vertical_slash_index_pooled,
    lines_of_blocks,
    query_aware_block_attention,
    query_aware_index,
    query_aware_index_rows,
    tiles_from_vertical_slash,
    tiles_from_query_aware,
    tiles_from_query_aware_rows,
    add_forced_and_min_budget,
    row_priority,
    apply_max_budget,
    select_head,
    select,
    sparse_attention_rows,
    sparse_attention_masked,
    dense_causal_attention,
)
