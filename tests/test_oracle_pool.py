"""The pooled oracle used by the full-size parity tests: a head split into row
ranges over worker processes gives the unsplit oracle's result."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from tests import oracle_pool as OP


@pytest.fixture(scope="module", autouse=True)
def _pool():
    yield
    OP.close_pool()


def test_row_ranges_cover_every_row_once():
    for T, parts in ((1, 4), (7, 3), (300, 16), (16384, 32)):
        rr = OP.row_ranges(T, parts)
        assert np.array_equal(np.concatenate(rr), np.arange(T))
        assert len(rr) <= parts


def test_split_equals_unsplit():
    rng = np.random.default_rng(5)
    T, D = 301, 16
    q, k, v, do = (rng.standard_normal((T, D)) for _ in range(4))
    lam = 0.3
    f0 = oracle.forward(q, k, v, lam, want_matrices=False)
    f1 = OP.forward_split(q, k, v, lam, parts=5)
    for n in ("Y", "M", "self_mass", "exch_mass", "LE"):
        np.testing.assert_allclose(f1[n], f0[n], rtol=1e-12, atol=1e-12)
    b0 = oracle.backward(q, k, v, lam, do)
    b1 = OP.backward_split(q, k, v, lam, do, parts=5)
    for n in ("dq", "dk", "dv", "dS"):
        np.testing.assert_allclose(b1[n], b0[n], rtol=1e-10, atol=1e-12)
    assert abs(b1["dlam"] - b0["dlam"]) <= 1e-10 * max(1.0, abs(b0["dlam"]))
    # per-head jobs match too
    Q, K, V, G = (a[None, None] for a in (q, k, v, do))
    (bh,) = OP.backward_heads(Q, K, V, lam, G, [(0, 0)])
    np.testing.assert_allclose(bh["dk"], b0["dk"], rtol=1e-12, atol=1e-12)
