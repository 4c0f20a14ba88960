"""CPU float64 oracle (test infrastructure only; see graphleap_ref)."""
from .graphleap_ref import (  # noqa: F401
    EPS, l2_normalize, pairwise_sq_dist, knn_order, knn_ref, knn_distances, dilated_lists,
    pool_keys_ref, max_pool_nodes_ref, max_relative_ref, mrconv_ref, mrconv_heads_ref, graph_source_blocks, stack_ref,
    VIG_PARAMS, gelu_ref, linear_ref, vig_block_ref, vig_stack_ref,
)
