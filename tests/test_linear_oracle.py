"""Pins of the Linear Relation oracle (CPU only): the recurrence against the
paper's unrolled sum, closed forms, strict historical support, finite
differences of the adjoint, and planted mistakes the pins must catch."""
import math
import os
import types

import numpy as np
import pytest

from oracle import linear_oracle

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "linear_oracle.py")


def _inputs(T, D, seed, gscale=0.3):
    rng = np.random.default_rng(seed)
    p1, p2, v, dY = (rng.standard_normal((T, D)) for _ in range(4))
    g = -np.abs(rng.standard_normal((T, D))) * gscale
    return p1, p2, v, g, dY


def check_unrolled(lo):
    """The recurrence equals the unrolled sum of App. A.4 (a different route:
    explicit per-pair retention products)."""
    for seed, (T, D) in enumerate([(7, 3), (10, 4)]):
        p1, p2, v, g, _ = _inputs(T, D, 10 + seed)
        a = lo.forward(p1, p2, v, g)["Y"]
        b = lo.forward_unrolled(p1, p2, v, g)
        assert np.allclose(a, b, atol=1e-13), "recurrence vs unrolled sum"


def check_closed_forms(lo):
    T, D = 9, 4
    p1, p2, v, g, _ = _inputs(T, D, 20)
    # no retention at all (alpha -> 0): history vanishes, Y = I~
    y = lo.forward(p1, p2, v, np.full((T, D), -800.0))["Y"]
    assert np.allclose(y, v, atol=1e-300), "alpha = 0"
    # T = 1: nothing historical
    assert np.array_equal(lo.forward(p1[:1], p2[:1], v[:1], g[:1])["Y"], v[:1])
    # full retention (g = 0) and identical unit coordinates e: the read of token t
    # is S_t sum_{j<t} S_j I~_j, whatever the direction of e
    e = np.zeros(D)
    e[1] = 3.0
    P = np.tile(e, (T, 1))
    out = lo.forward(P, P, v, np.zeros((T, D)))
    S = 1.0 / (1.0 + math.exp(-(9.0 / 2.0) / 2.0))            # p1 . p2 = 9, d_h = 4, tau_S = 2
    assert np.allclose(out["S"], S, atol=1e-15)
    for t in range(T):
        assert np.allclose(out["Y"][t], v[t] + S * S * v[:t].sum(axis=0), atol=1e-13), f"g = 0, t = {t}"
    # orthogonal coordinates: ^p2_j . ^p1_t = 0 means no Exchange at all
    P1 = np.tile(np.eye(D)[0], (T, 1))
    P2 = np.tile(np.eye(D)[1], (T, 1))
    assert np.allclose(lo.forward(P1, P2, v, g)["Y"], v, atol=1e-15)


def check_strictly_historical(lo):
    """E_t reads the state before token t is written: changing I~ of tokens
    from t on, or p2 and g of later tokens, leaves Y_t - I~_t unchanged (p2_t
    itself enters E_t through S_t)."""
    T, D = 8, 3
    p1, p2, v, g, _ = _inputs(T, D, 30)
    base = lo.forward(p1, p2, v, g)["Y"]
    t = 5
    v2, p22, g2 = v.copy(), p2.copy(), g.copy()
    v2[t:] += 1.0
    p22[t + 1:] *= -2.0
    g2[t + 1:] -= 0.5
    alt = lo.forward(p1, p22, v2, g2)["Y"]
    assert np.allclose((alt - v2)[: t + 1], (base - v)[: t + 1], atol=1e-14), "strict history"
    # retention of token t itself does act on token t's read (C_t^- = D_t C_{t-1})
    g3 = g.copy()
    g3[t] -= 1.0
    assert not np.allclose(lo.forward(p1, p2, v, g3)["Y"][t], base[t])


def check_gradients_fd(lo):
    h = 1e-6
    for seed, (T, D) in enumerate([(6, 3), (5, 4)]):
        p1, p2, v, g, dY = _inputs(T, D, 40 + seed, gscale=0.5)
        r = lo.backward(p1, p2, v, g, dY)
        loss = lambda a, b, c, d: float(np.sum(dY * lo.forward(a, b, c, d)["Y"]))
        for name, X in (("dp1", p1), ("dp2", p2), ("dv", v), ("dg", g)):
            num = np.empty_like(X)
            for idx in np.ndindex(X.shape):
                old = X[idx]
                X[idx] = old + h
                lp = loss(p1, p2, v, g)
                X[idx] = old - h
                lm = loss(p1, p2, v, g)
                X[idx] = old
                num[idx] = (lp - lm) / (2 * h)
            assert np.allclose(r[name], num, atol=3e-8), f"{name} vs FD"


def check_gate_closed_forms(lo):
    """Eq. 15 at points where softplus is known: softplus(0) = ln 2, softplus(x)
    tends to x for large x and to e^x for very negative x; g < 0 everywhere
    and alpha = exp(g) in (0, 1]; A_log scales g by e^A_log."""
    D = 4
    a = np.array([0.0, 1.0, -2.0, 0.5])
    b = np.array([0.3, -0.3, 1.5, -1.5])
    r0 = np.tile(-b, (3, 1))                                 # r + dt_bias = 0
    assert np.allclose(lo.kda_gate(r0, a, b), -np.exp(a) * math.log(2.0), atol=1e-15), "softplus(0)"
    big = np.full((1, D), 40.0) - b
    assert np.allclose(lo.kda_gate(big, a, b), -np.exp(a) * 40.0, rtol=1e-15), "softplus(40) = 40"
    small = np.full((1, D), -40.0) - b
    assert np.allclose(lo.kda_gate(small, a, b), -np.exp(a) * math.exp(-40.0), rtol=1e-12), "softplus(-40)"
    rng = np.random.default_rng(60)
    r = rng.standard_normal((50, D)) * 5.0
    g = lo.kda_gate(r, a, b)
    assert np.all(g < 0.0) and np.all(np.exp(g) <= 1.0), "g < 0, alpha in (0, 1]"
    assert np.allclose(lo.kda_gate(r, a + 1.0, b), math.e * g, rtol=1e-14), "A_log scales by e^A_log"


def check_gate_gradients_fd(lo):
    """The chain through eq. 15 and the recurrence: dr, dA_log and ddt_bias from
    kda_gate_backward (fed dg from the recurrence's adjoint) against central
    differences of sum(dY * Y) with g = kda_gate(r, A_log, dt_bias)."""
    h = 1e-6
    T, D = 6, 3
    p1, p2, v, _, dY = _inputs(T, D, 70)
    rng = np.random.default_rng(71)
    r = rng.standard_normal((T, D))
    a = rng.standard_normal(D) * 0.5
    b = rng.standard_normal(D) * 0.5
    dg = lo.backward(p1, p2, v, lo.kda_gate(r, a, b), dY)["dg"]
    got = lo.kda_gate_backward(r, a, b, dg)
    loss = lambda: float(np.sum(dY * lo.forward(p1, p2, v, lo.kda_gate(r, a, b))["Y"]))
    for name, X in (("dr", r), ("da_log", a), ("ddt_bias", b)):
        num = np.empty_like(X)
        for idx in np.ndindex(X.shape):
            old = X[idx]
            X[idx] = old + h
            lp = loss()
            X[idx] = old - h
            lm = loss()
            X[idx] = old
            num[idx] = (lp - lm) / (2 * h)
        assert np.allclose(got[name], num, atol=3e-8), f"{name} vs FD"


ALL_CHECKS = [check_unrolled, check_closed_forms, check_strictly_historical, check_gradients_fd,
              check_gate_closed_forms, check_gate_gradients_fd]


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda c: c.__name__)
def test_pin(check):
    check(linear_oracle)


MUTATIONS = [
    ("read_after_write", "        Y[t] = v[t] + S[t] * (Cm.T @ h1)",
     "        Y[t] = v[t] + S[t] * ((Cm + S[t] * np.outer(h2, v[t])).T @ h1)"),
    ("retention_skips_current", "        Cm = np.exp(g[t])[:, None] * C                        #",
     "        Cm = C                        #"),
    ("write_unnormalised", "        h2 = p2[t] / np.linalg.norm(p2[t])", "        h2 = p2[t]"),
    ("self_drops_tau", "        S[t] = expit(s * float(p1[t] @ p2[t]) / tau_s)        # Ask Self",
     "        S[t] = expit(s * float(p1[t] @ p2[t]))        # Ask Self"),
    ("state_transposed_read", "        Y[t] = v[t] + S[t] * (Cm.T @ h1)", "        Y[t] = v[t] + S[t] * (Cm @ h1)"),
    ("adjoint_dg_sign", "        dg[t] = a * np.sum(dCm * Cs[t], axis=1)", "        dg[t] = -a * np.sum(dCm * Cs[t], axis=1)"),
    ("adjoint_norm_projection", "        dp1[t] += (dh1 - h1[t] * float(h1[t] @ dh1)) / n1[t]",
     "        dp1[t] += dh1 / n1[t]"),
    ("adjoint_write_transposed", "        dv[t] = S[t] * (dC.T @ h2[t]) + dY[t]", "        dv[t] = S[t] * (dC @ h2[t]) + dY[t]"),
    ("gate_drops_bias", "    softplus = np.logaddexp(0.0, r + dt_bias)", "    softplus = np.logaddexp(0.0, r)"),
    ("gate_exp_of_softplus", "    return -np.exp(a_log) * softplus", "    return -np.exp(a_log * softplus)"),
    ("gate_adjoint_softplus_for_sigmoid", "    dr = dg * (-np.exp(a_log) * expit(r + dt_bias))",
     "    dr = dg * (-np.exp(a_log) * np.logaddexp(0.0, r + dt_bias))"),
    ("gate_adjoint_alog_drops_dg", "np.sum(dg * kda_gate(r, a_log, dt_bias), axis=lead)",
     "np.sum(kda_gate(r, a_log, dt_bias), axis=lead)"),
]


def _load_mutant(old, new):
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation anchor must occur once: {old!r}"
    mod = types.ModuleType("linear_oracle_mutant")
    mod.__file__ = SRC
    exec(compile(text.replace(old, new), SRC + " (mutant)", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mutation_is_caught(name, old, new):
    mod = _load_mutant(old, new)
    caught = []
    for check in ALL_CHECKS:
        try:
            check(mod)
        except (AssertionError, ValueError, IndexError, FloatingPointError):
            caught.append(check.__name__)
    assert caught, f"planted mistake {name} passed every pin"
