"""FlashRelation on MI355X (gfx950): the exact causal Full Relation operator.

The operator runs in librelation.so (hand-written HIP kernels behind a C ABI,
see include/relation.h); ``paper_2608_20172_amd.binding`` is its ctypes
binding. Importing the package does not load the library; the first call does,
and raises if the library has not been built.
"""
from .binding import (  # noqa: F401
    relation,
    relation_fwd,
    relation_bwd,
    relation_bwd_workspace_bytes,
    relation_fwd_materialized,
    relation_fwd_materialized_workspace_bytes,
    relation_exchange_allocation,
    load_library,
    TAU_S,
)
