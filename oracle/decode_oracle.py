"""fp64 CPU oracle for one decode step of the causal Full Relation operator and
for the running Exchange statistics that a split (or sharded) key scan merges.

TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
baseline leg may import this module. The product path never calls it, and it
shares no code with that path.

A decode step computes the one new row of the operator: the new token sits at
one-based position i = L of its sequence, its own key and value are entry L of
the cache (the Self entry, eq. 2), and entries 1 .. L-1 are its history (the
Exchange entries, with the count correction -lambda ln i taken at the
absolute position i). The row is exactly row i of the full forward pass
(relation_oracle.forward), which is what ``decode_step`` evaluates.

``exchange_state`` gives, for one query row and a set of its historical keys,
the statistics the FlashRelation scan carries (eq. 11): m = max_j E_ij,
l = sum_j exp(E_ij - m), z = sum_j exp(E_ij - m) v_j, with E_ij = SiLU(U_ij) the
Exchange map before the count correction. Any partition of the history into
key sets gives states whose merge (App. A.3: rescale to the common maximum and
add) is the state of the whole history; the epilogue of eqs. 12-13 then joins
Self and lambda.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import expit

from .relation_oracle import TAU_S, forward

__all__ = ["decode_step", "exchange_state"]


def decode_step(q_new, k_cache, v_cache, L: int, lam: float, *, tau_s: float = TAU_S, scale=None):
    """y [D] and M (= ln Z + lambda ln i) of the new token at position i = L,
    against cache entries 1 .. L (fp64 [Tmax, D] arrays; entry L is its own)."""
    q_new = np.asarray(q_new, np.float64)
    D = q_new.shape[-1]
    q = np.zeros((L, D))
    q[L - 1] = q_new
    f = forward(q, k_cache[:L], v_cache[:L], lam, tau_s=tau_s, scale=scale, want_matrices=False,
                rows=np.array([L - 1]))
    return f["Y"][0], float(f["M"][0])


def exchange_state(q_i, k, v, keys, *, scale=None):
    """(m, l, z) over the listed zero-based historical keys of one query row."""
    q_i = np.asarray(q_i, np.float64)
    D = q_i.shape[-1]
    s = 1.0 / math.sqrt(D) if scale is None else float(scale)
    keys = np.asarray(keys, dtype=np.int64)
    if keys.size == 0:
        return -math.inf, 0.0, np.zeros(D)
    U = s * (np.asarray(k, np.float64)[keys] @ q_i)      # eq. (1)
    E = U * expit(U)                                     # eq. (2), Exchange map
    m = float(E.max())
    w = np.exp(E - m)
    return m, float(w.sum()), w @ np.asarray(v, np.float64)[keys]
