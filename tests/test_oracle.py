"""Pins of the fp64 oracle (CPU only). See oracle_pins.py for what each pins."""
import math
import os

import numpy as np
import pytest

import oracle
from tests import oracle_pins as pins


@pytest.mark.parametrize("check", pins.ALL_CHECKS, ids=lambda c: c.__name__)
def test_pin(check):
    check(oracle)


def test_zero_keys_closed_form_long_rows():
    """K = 0 closed form at long context: the oracle row-blocked up to T = 2048
    matches the closed form, and the closed form at T = 16384 lies where the
    count correction puts it (g grows towards 1 as the history grows for lambda < 1)."""
    T, D = 2048, 4
    rng = np.random.default_rng(3)
    q = rng.standard_normal((T, D))
    v = rng.standard_normal((T, D))
    f = oracle.forward(q, np.zeros((T, D)), v, 0.5, want_matrices=False, row_block=512)
    for i in (2, 3, 128, 2048):
        assert abs(f["exch_mass"][i - 1] - pins.closed_form_zero_keys_g(i, 0.5)) < 1e-14
    g = [pins.closed_form_zero_keys_g(i, 0.5) for i in (2, 3, 128, 2048, 16384)]
    assert all(a < b for a, b in zip(g, g[1:])) and g[-1] < 1.0
    assert abs(g[0] - 1 / (1 + math.exp(0.5) * math.sqrt(2))) < 1e-15


def test_parameter_budget_table6():
    """Table 6: Relation - MHA = layers * (1 + H/2): lambda is the only learnable
    Self/Exchange parameter, so the operator's parameter argument is lambda alone."""
    path = os.path.join(os.path.dirname(__file__), "golden", "table6_param_counts.txt")
    rows = [ln.split() for ln in open(path) if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 3
    for _, L, H, mha, rel in rows:
        L, H, mha, rel = int(L), int(H), int(mha), int(rel)
        assert rel - mha == L * (1 + H // 2)


def test_batched_sum_of_heads():
    B, H, T, D = 2, 3, 17, 4
    rng = np.random.default_rng(8)
    q, k, v, dO = (rng.standard_normal((B, H, T, D)) for _ in range(4))
    fb = oracle.forward_batched(q, k, v, 0.5)
    bb = oracle.backward_batched(q, k, v, 0.5, dO)
    tot = 0.0
    for b in range(B):
        for h in range(H):
            f = oracle.forward(q[b, h], k[b, h], v[b, h], 0.5)
            assert np.allclose(fb["Y"][b, h], f["Y"], atol=0)
            tot += oracle.backward(q[b, h], k[b, h], v[b, h], 0.5, dO[b, h])["dlam"]
    assert abs(bb["dlam"] - tot) < 1e-12
