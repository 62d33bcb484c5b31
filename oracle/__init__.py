"""CPU oracle for the DominoTree draft-tree builder.

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.
"""
from .dominotree_ref import (  # noqa: F401
    DT_BF16,
    DT_F32,
    NORM_SLICE,
    NORM_TAIL,
    SCORER_COND,
    SCORER_HEAD,
    SCORER_MARG,
    SCORER_STATIC,
    TREE_NONFINITE,
    build_tree,
    build_trees,
    effective_temperature,
    gru_cell,
    logsumexp,
    scan,
    scan_row,
    silu,
    score_paths,
    widen,
)
