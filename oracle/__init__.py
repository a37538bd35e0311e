"""SparSTAR CPU oracle (test infrastructure only; never imported by the product path).

See sparstar_oracle.py for the statement of what each function computes and the
passage of the paper it follows.
"""
from .sparstar_oracle import (  # noqa: F401
    block_scores,
    block_token_range,
    budget_k,
    dense_attention,
    keep_blocks,
    keep_ranges_for_clip,
    num_blocks,
    partition,
    pool,
    retained_mass,
    retained_support,
    scale_densities,
    segment_blocks,
    select,
    selectable_blocks,
    sparse_attention,
    token_mask,
    token_topk_mass,
    topk_idx,
)
