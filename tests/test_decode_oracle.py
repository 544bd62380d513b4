"""Pins of the decode oracle (CPU only): the decode row against closed forms
and the operator's own definition checked by brute force, and the Exchange
states against their definition and their merge."""
import math

import numpy as np
import pytest

import oracle
from oracle import decode_oracle as DO
from tests import oracle_pins


def _cache(Tmax, D, seed, std=1.0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(D) * std, rng.standard_normal((Tmax, D)) * std,
            rng.standard_normal((Tmax, D)))


@pytest.mark.parametrize("L", [1, 2, 5, 9])
def test_decode_row_brute_force(L):
    """The decode row equals the last row of the pure-Python brute force of
    eqs. (1)-(3) on the sequence whose last query is the new token."""
    qn, K, V = _cache(12, 3, seed=L, std=1.3)
    lam = 0.6
    y, M = DO.decode_step(qn, K, V, L, lam)
    q = np.zeros((L, 3))
    q[L - 1] = qn
    Yb, _ = oracle_pins.brute_force_forward(q.tolist(), K[:L].tolist(), V[:L].tolist(), lam)
    assert np.allclose(y, Yb[L - 1], atol=1e-13)


def test_decode_first_token_and_zero_keys():
    qn, K, V = _cache(8, 4, seed=3)
    # one token: pure Self, y = v_1
    y, M = DO.decode_step(qn, K, V, 1, 0.5)
    assert np.array_equal(y, V[0])
    # all historical keys zero: E = 0, so the Exchange part is the plain mean of
    # v_1..v_{i-1} and g = (i-1) i^-lambda / ((i-1) i^-lambda + e^{S_i}) with
    # S_i = sigmoid(U_ii / 2)
    L, lam = 6, 0.5
    K2 = K.copy()
    K2[: L - 1] = 0.0
    y, M = DO.decode_step(qn, K2, V, L, lam)
    u = float(qn @ K2[L - 1]) / 2.0
    S = 1.0 / (1.0 + math.exp(-u / 2.0))
    ex = (L - 1) * L ** (-lam)
    g = ex / (ex + math.exp(S))
    want = (1 - g) * V[L - 1] + g * V[: L - 1].mean(axis=0)
    assert np.allclose(y, want, atol=1e-14)
    # M = ln Z + lambda ln i with Z = (i-1) i^-lambda + e^S
    assert abs(M - (math.log(ex + math.exp(S)) + lam * math.log(L))) < 1e-13


def test_exchange_state_single_key_and_empty():
    qn, K, V = _cache(6, 4, seed=5)
    m, l, z = DO.exchange_state(qn, K, V, [2])
    u = float(qn @ K[2]) / 2.0
    assert abs(m - u / (1.0 + math.exp(-u))) < 1e-15 and l == 1.0 and np.array_equal(z, V[2])
    m, l, z = DO.exchange_state(qn, K, V, [])
    assert m == -math.inf and l == 0.0 and not z.any()


def test_exchange_states_merge_to_the_row():
    """States of any partition of the history, merged by rescaling to the common
    maximum, give L^E = m + ln l and the Exchange mean z / l of the whole row as
    the operator oracle computes them (logsumexp and pi over the full matrix)."""
    qn, K, V = _cache(40, 8, seed=7, std=1.5)
    L = 37
    q = np.zeros((L, 8))
    q[L - 1] = qn
    f = oracle.forward(q, K[:L], V[:L], 0.3, rows=np.array([L - 1]))
    Ibar = f["pi"][0] @ V[:L]
    rng = np.random.default_rng(1)
    for nparts in (1, 2, 5):
        cuts = np.sort(rng.choice(np.arange(1, L - 1), size=nparts - 1, replace=False)) if nparts > 1 else []
        parts = np.split(np.arange(L - 1), cuts)
        st = [DO.exchange_state(qn, K, V, p) for p in parts]
        m = max(s[0] for s in st)
        l = sum(s[1] * math.exp(s[0] - m) for s in st)
        z = sum(s[2] * math.exp(s[0] - m) for s in st)
        assert abs(m + math.log(l) - f["LE"][0]) < 1e-12
        assert np.allclose(z / l, Ibar, atol=1e-12)
