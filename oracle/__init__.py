"""fp64 CPU oracle for the causal Full Relation operator.

TEST INFRASTRUCTURE: only tests, the smoke check and the benchmark's CPU
baseline import this package; the product path never does.
"""
from .relation_oracle import forward, backward, forward_batched, backward_batched, TAU_S  # noqa: F401
