"""Seeded synthetic inputs for tree-ensemble prediction.

This module only draws random numbers and lays out forest arrays; it holds none
of the prediction arithmetic.  Both the CPU oracle (tests, CPU baseline) and the
HIP path consume exactly the arrays produced here.
"""
from .forests import (  # noqa: F401
    AGG_SUM, AGG_MEAN, XFORM_IDENTITY, XFORM_SIGMOID, XFORM_SOFTMAX,
    Forest, Workload, CONFIGS, EXTRA_CONFIGS, make_workload, make_forest, x_rows, x_rows_threaded, x_block, x_take,
    permute_nodes, random_tiny_forest, perfect_tree_arrays, concat_trees, with_vector_leaves,
    BLOCK_ROWS,
)
