"""fp64 CPU oracle for the causal Full Relation operator, the steps around it
in a layer (RoPE on the relation projections, Givens head-pair mixing), one
decode step with the Exchange states a split key scan merges, and Linear
Relation (the recurrent-state Exchange).

TEST INFRASTRUCTURE: only tests, the smoke check and the benchmark's CPU
baseline import this package; the product path never does.
"""
from .relation_oracle import forward, backward, forward_batched, backward_batched, TAU_S  # noqa: F401
from . import layer_oracle  # noqa: F401
from . import decode_oracle  # noqa: F401
from . import linear_oracle  # noqa: F401
