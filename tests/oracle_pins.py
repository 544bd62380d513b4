"""Checks that pin the fp64 oracle to facts fixed by the paper and by
mathematics, independently of the oracle's own code.

Each ``check_*`` takes the oracle module under test and raises AssertionError
on a mismatch. ``test_oracle.py`` runs them on the real oracle, and
``test_oracle_mutations.py`` runs them on copies of the oracle with planted
mistakes, to show that every planted mistake is caught by at least one pin.
"""
from __future__ import annotations

import math

import numpy as np

TAU = 2.0


def _rand(T, D, seed, std=1.0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((T, D)) * std, rng.standard_normal((T, D)) * std,
            rng.standard_normal((T, D)), rng.standard_normal((T, D)))


# ---------------------------------------------------------------------------
# 1. Brute force from the definition, pure Python floats, tiny T
# ---------------------------------------------------------------------------
def brute_force_forward(q, k, v, lam, tau=TAU):
    """Eq. (1)-(3) evaluated entry by entry with the math module. Returns Y and
    the flow matrix F as nested lists."""
    T, D = len(q), len(q[0])
    s = 1.0 / math.sqrt(D)
    F = [[0.0] * T for _ in range(T)]
    Y = [[0.0] * D for _ in range(T)]
    for i in range(T):
        logits = []
        for j in range(i + 1):
            u = s * sum(q[i][d] * k[j][d] for d in range(D))
            if j == i:
                logits.append(1.0 / (1.0 + math.exp(-u / tau)))
            else:
                silu = u / (1.0 + math.exp(-u))
                logits.append(silu - lam * math.log(i + 1))
        mx = max(logits)
        w = [math.exp(x - mx) for x in logits]
        z = sum(w)
        for j in range(i + 1):
            F[i][j] = w[j] / z
            for d in range(D):
                Y[i][d] += F[i][j] * v[j][d]
    return Y, F


def check_brute_force(orc):
    for seed, (T, D, lam) in enumerate([(6, 3, 0.5), (9, 4, -0.7), (5, 2, 1.3)]):
        q, k, v, _ = _rand(T, D, 100 + seed)
        Yb, Fb = brute_force_forward(q.tolist(), k.tolist(), v.tolist(), lam)
        f = orc.forward(q, k, v, lam)
        assert np.allclose(f["Y"], np.array(Yb), rtol=0, atol=1e-13), "Y vs brute force"
        assert np.allclose(f["F"], np.array(Fb), rtol=0, atol=1e-13), "F vs brute force"


# ---------------------------------------------------------------------------
# 2. Invariants stated by the paper (eqs. 5-10, App. A.1.2-A.1.8)
# ---------------------------------------------------------------------------
def check_invariants(orc):
    from scipy.special import logsumexp
    T, D = 37, 8
    for seed, lam in [(1, 0.5), (2, 0.0), (3, -1.0), (4, 2.0)]:
        q, k, v, _ = _rand(T, D, seed, std=1.5)
        f = orc.forward(q, k, v, lam)
        F, pi, g, sm = f["F"], f["pi"], f["exch_mass"], f["self_mass"]
        i1 = np.arange(1, T + 1)
        # rows of F sum to one, F is causal
        assert np.allclose(F.sum(1), 1.0, atol=1e-13), "F rows sum"
        assert np.all(np.triu(F, 1) == 0.0), "F causal"
        # Self mass + Exchange mass = 1 (eq. 6)
        assert np.allclose(sm + g, 1.0, atol=1e-13), "F_ii + g_i = 1"
        assert np.allclose(sm, np.diag(F), atol=0), "self mass is the diagonal"
        # boundary row (App. A.1.8)
        assert sm[0] == 1.0 and g[0] == 0.0 and np.array_equal(f["Y"][0], v[0]), "row 1"
        assert f["LE"][0] == -np.inf
        # allocation sums to one and factorises F (eq. 7)
        assert np.allclose(pi[1:].sum(1), 1.0, atol=1e-13), "pi rows sum"
        low = np.tril(np.ones((T, T), bool), -1)
        assert np.allclose(F[low], (g[:, None] * pi)[low], atol=1e-14), "F = g pi"
        # L^E from the Exchange entries by an independent logsumexp on E restricted to j < i
        E = f["E"]
        LE = np.array([logsumexp(E[i, :i]) if i else -np.inf for i in range(T)])
        assert np.allclose(f["LE"][1:], LE[1:], atol=1e-12), "L^E"
        # odds identity log(g/F_ii) = A - S (eq. 9)
        A = LE - lam * np.log(i1)
        assert np.allclose(np.log(g[1:] / sm[1:]), (A - f["S"])[1:], atol=1e-11), "odds"
        # g = sigmoid(A - S) computed without the matrix
        assert np.allclose(g[1:], 1 / (1 + np.exp(f["S"][1:] - A[1:])), atol=1e-13)
        # information-space form (eq. 8): Y = (1-g) I~ + g Ibar
        Ibar = pi @ v
        assert np.allclose(f["Y"], (1 - g)[:, None] * v + g[:, None] * Ibar, atol=1e-12), "eq. 8"
        # saved statistic: F_ij = exp(E_ij - M_i) below the diagonal, F_ii = exp(S_i - M_i + lam log i)
        M = f["M"]
        assert np.allclose(F[low], np.exp(E - M[:, None])[low], atol=1e-13), "F via M"
        assert np.allclose(sm, np.exp(f["S"] - M + lam * np.log(i1)), atol=1e-13)
    # lambda shifts only the Self-Exchange split, never the allocation (eq. 10)
    q, k, v, _ = _rand(T, D, 9, std=1.5)
    p1 = orc.forward(q, k, v, 0.5)["pi"]
    p2 = orc.forward(q, k, v, -1.7)["pi"]
    assert np.allclose(p1, p2, atol=1e-14), "pi independent of lambda"
    assert not np.allclose(orc.forward(q, k, v, 0.5)["exch_mass"],
                           orc.forward(q, k, v, -1.7)["exch_mass"]), "g depends on lambda"


# ---------------------------------------------------------------------------
# 3. The tiled online Exchange scan of FlashRelation (eqs. 11-13, App. A.3)
#    reaches the Full Relation output exactly (App. A.3.5)
# ---------------------------------------------------------------------------
def flash_scan_row(u_row, s_i, v, i, lam, tiles):
    """One query row i (zero-based) by the tiled scan: Exchange entries only
    in (m, l, z), Self joins in the epilogue."""
    m, l, z = -np.inf, 0.0, np.zeros(v.shape[1])
    for j0, j1 in tiles:
        j1 = min(j1, i)
        if j0 >= j1:
            continue
        e = u_row[j0:j1] / (1 + np.exp(-u_row[j0:j1]))
        mp = max(m, e.max())
        w = np.exp(e - mp)
        l = math.exp(m - mp) * l + w.sum()
        z = math.exp(m - mp) * z + w @ v[j0:j1]
        m = mp
    S = 1 / (1 + math.exp(-u_row[i] / TAU))
    if l == 0.0:
        return v[i].copy(), 0.0
    A = m + math.log(l) - lam * math.log(i + 1)
    g = 1 / (1 + math.exp(S - A))
    return (1 - g) * v[i] + g * z / l, g


def check_flash_scan(orc):
    rng = np.random.default_rng(5)
    for T, D, lam, std in [(50, 8, 0.5, 3.0), (33, 4, -0.3, 6.0)]:
        q, k, v, _ = _rand(T, D, int(rng.integers(1000)), std=std)
        s = 1.0 / math.sqrt(D)
        f = orc.forward(q, k, v, lam)
        cuts = np.sort(rng.choice(np.arange(1, T), size=6, replace=False))
        edges = [0, *cuts.tolist(), T]
        tiles = list(zip(edges[:-1], edges[1:]))
        for i in range(T):
            u_row = s * (k @ q[i])
            y, g = flash_scan_row(u_row, s * q[i] @ k[i], v, i, lam, tiles)
            assert np.allclose(y, f["Y"][i], atol=1e-12), f"flash scan row {i}"
            assert abs(g - f["exch_mass"][i]) < 1e-12


# ---------------------------------------------------------------------------
# 4. Closed forms
# ---------------------------------------------------------------------------
def closed_form_zero_keys_g(i, lam):
    """K = 0: U = 0, so S_i = 1/2, E = 0, and the row normaliser is
    e^{1/2} + (i - 1) i^{-lambda}; g_i is the Exchange share of it."""
    x = (i - 1) * i ** (-lam)
    return x / (x + math.exp(0.5))


def check_closed_forms(orc):
    # K = 0
    T, D = 64, 4
    rng = np.random.default_rng(11)
    q = rng.standard_normal((T, D))
    v = rng.standard_normal((T, D))
    k = np.zeros((T, D))
    for lam in (0.5, 0.0, -0.8):
        f = orc.forward(q, k, v, lam)
        g = np.array([closed_form_zero_keys_g(i, lam) for i in range(1, T + 1)])
        assert np.allclose(f["exch_mass"], g, atol=1e-14), "K=0 g"
        mean_hist = np.vstack([np.zeros(D), np.cumsum(v, 0)[:-1] / np.arange(1, T)[:, None]])
        Y = (1 - g)[:, None] * v + g[:, None] * mean_hist
        assert np.allclose(f["Y"], Y, atol=1e-13), "K=0 Y"
        assert np.allclose(f["S"], 0.5)
    # all keys equal: pi uniform, L^E_i = SiLU(u_i) + ln(i - 1)
    kk = rng.standard_normal(D) * 2
    k = np.tile(kk, (T, 1))
    q = rng.standard_normal((T, D)) * 2
    lam = 0.3
    f = orc.forward(q, k, v, lam)
    u = (q @ kk) / math.sqrt(D)
    silu = u / (1 + np.exp(-u))
    i1 = np.arange(1, T + 1)
    LE = silu[1:] + np.log(i1[1:] - 1)
    assert np.allclose(f["LE"][1:], LE, atol=1e-12), "equal keys L^E"
    S = 1 / (1 + np.exp(-u / TAU))
    g = 1 / (1 + np.exp(S[1:] - (LE - lam * np.log(i1[1:]))))
    assert np.allclose(f["exch_mass"][1:], g, atol=1e-13), "equal keys g"
    # V constant: Y = c whatever Q, K, lambda
    q, k, _, dO = _rand(T, D, 12, std=2.0)
    c = rng.standard_normal(D)
    vc = np.tile(c, (T, 1))
    f = orc.forward(q, k, vc, 0.7)
    assert np.allclose(f["Y"], vc, atol=1e-13), "V constant"
    # T = 1
    q1, k1, v1, d1 = _rand(1, D, 13)
    f = orc.forward(q1, k1, v1, 0.5)
    assert np.array_equal(f["Y"], v1) and f["exch_mass"][0] == 0.0


def check_lambda_limits(orc):
    T, D = 24, 4
    q, k, v, _ = _rand(T, D, 14)
    f = orc.forward(q, k, v, 60.0)             # lambda -> +inf: history suppressed
    assert np.max(f["exch_mass"]) < 1e-15 and np.allclose(f["Y"], v, atol=1e-14)
    f = orc.forward(q, k, v, -60.0)            # lambda -> -inf: Self suppressed (rows > 1)
    assert np.min(f["exch_mass"][1:]) > 1 - 1e-15
    Ibar = f["pi"] @ v
    assert np.allclose(f["Y"][1:], Ibar[1:], atol=1e-13)


# ---------------------------------------------------------------------------
# 5. Gradients: central finite differences and the two analytic routes
# ---------------------------------------------------------------------------
def _loss(orc, q, k, v, lam, dO):
    return float((orc.forward(q, k, v, lam, want_matrices=False)["Y"] * dO).sum())


def check_gradients_fd(orc):
    h = 1e-6
    for T, D, lam, seed in [(9, 4, 0.5, 21), (7, 3, -1.2, 22)]:
        q, k, v, dO = _rand(T, D, seed, std=1.3)
        for route in ("softmax", "factorised"):
            r = orc.backward(q, k, v, lam, dO, route=route)
            for name, X in (("dq", q), ("dk", k), ("dv", v)):
                num = np.empty_like(X)
                for idx in np.ndindex(X.shape):
                    old = X[idx]
                    X[idx] = old + h
                    lp = _loss(orc, q, k, v, lam, dO)
                    X[idx] = old - h
                    lm = _loss(orc, q, k, v, lam, dO)
                    X[idx] = old
                    num[idx] = (lp - lm) / (2 * h)
                assert np.allclose(r[name], num, atol=2e-8), f"{route} {name} vs FD"
            num_l = (_loss(orc, q, k, v, lam + h, dO) - _loss(orc, q, k, v, lam - h, dO)) / (2 * h)
            assert abs(r["dlam"] - num_l) < 2e-8, f"{route} dlam vs FD"


def check_routes_agree(orc):
    T, D = 40, 8
    q, k, v, dO = _rand(T, D, 31, std=1.7)
    a = orc.backward(q, k, v, 0.4, dO, route="softmax")
    b = orc.backward(q, k, v, 0.4, dO, route="factorised")
    for n in ("dq", "dk", "dv", "dS"):
        scale = max(1.0, np.abs(a[n]).max())
        assert np.abs(a[n] - b[n]).max() <= 1e-12 * scale, f"routes {n}"
    assert abs(a["dlam"] - b["dlam"]) <= 1e-12 * max(1.0, abs(a["dlam"])), "routes dlam"


def check_gradient_special_cases(orc):
    T, D = 20, 4
    q, k, _, dO = _rand(T, D, 41, std=1.5)
    rng = np.random.default_rng(42)
    vc = np.tile(rng.standard_normal(D), (T, 1))
    r = orc.backward(q, k, vc, 0.5, dO)
    # Y does not depend on Q, K, lambda when V is constant
    assert np.abs(r["dq"]).max() < 1e-12 and np.abs(r["dk"]).max() < 1e-12
    assert abs(r["dlam"]) < 1e-12
    # rows of F sum to one, so the columns of dV add up to the rows of dO
    q, k, v, dO = _rand(T, D, 43, std=1.5)
    r = orc.backward(q, k, v, 0.5, dO)
    assert np.allclose(r["dv"].sum(0), dO.sum(0), atol=1e-12), "sum dV = sum dO"
    # T = 1: Y = V
    q1, k1, v1, d1 = _rand(1, D, 44)
    r = orc.backward(q1, k1, v1, 0.5, d1)
    assert np.array_equal(r["dv"], d1) and not r["dq"].any() and not r["dk"].any()
    assert r["dlam"] == 0.0


def check_row_blocking(orc):
    T, D = 45, 8
    q, k, v, dO = _rand(T, D, 51, std=1.5)
    a = orc.forward(q, k, v, 0.5, want_matrices=False)
    b = orc.forward(q, k, v, 0.5, want_matrices=False, row_block=7)
    for n in ("Y", "exch_mass", "self_mass", "LE", "M"):
        assert np.allclose(a[n], b[n], atol=1e-14, equal_nan=True), f"blocked {n}"
    ra = orc.backward(q, k, v, 0.5, dO)
    rb = orc.backward(q, k, v, 0.5, dO, row_block=7)
    for n in ("dq", "dk", "dv", "dS"):
        assert np.allclose(ra[n], rb[n], atol=1e-13), f"blocked {n}"
    assert abs(ra["dlam"] - rb["dlam"]) < 1e-12
    # a subset of rows gives the same rows; rows {j0..T-1} give complete dk, dv for keys >= j0
    sub = np.array([0, 3, 17, 30, 44])
    c = orc.forward(q, k, v, 0.5, want_matrices=False, rows=sub, row_block=2)
    for n in ("Y", "exch_mass", "M"):
        assert np.allclose(c[n], a[n][sub], atol=1e-14, equal_nan=True), f"row subset {n}"
    j0 = 30
    rc = orc.backward(q, k, v, 0.5, dO, rows=np.arange(j0, T), row_block=4)
    assert np.allclose(rc["dq"], ra["dq"][j0:], atol=1e-13), "row subset dq"
    assert np.allclose(rc["dk"][j0:], ra["dk"][j0:], atol=1e-13), "row subset dk"
    assert np.allclose(rc["dv"][j0:], ra["dv"][j0:], atol=1e-13), "row subset dv"
    assert np.allclose(rc["dS"], ra["dS"][j0:], atol=1e-13), "row subset dS"


# ---------------------------------------------------------------------------
# 7. Exchange-only transport (App. D, ablation definitions): the same flow F,
#    Y_i = sum_{j<i} F_ij I~_j, historical weights not renormalised
# ---------------------------------------------------------------------------
def check_exchange_only(orc):
    for seed, (T, D, lam) in enumerate([(6, 3, 0.5), (8, 2, -0.9)]):
        q, k, v, dO = _rand(T, D, 300 + seed, std=1.4)
        # brute force: F from the pure-Python definition, the historical part transported
        _, Fb = brute_force_forward(q.tolist(), k.tolist(), v.tolist(), lam)
        Yb = [[sum(Fb[i][j] * v[j][d] for j in range(i)) for d in range(D)] for i in range(T)]
        f = orc.forward(q, k, v, lam, transport="exchange")
        assert np.allclose(f["Y"], np.array(Yb), rtol=0, atol=1e-13), "exchange-only Y vs brute force"
        assert not f["Y"][0].any(), "row 1 transports nothing"
        # the flow itself is the full operator's
        g = orc.forward(q, k, v, lam)
        assert np.allclose(f["F"], g["F"], atol=0) and np.allclose(f["exch_mass"], g["exch_mass"], atol=0)
        # central differences of sum(dO * Y) for every input entry and lambda
        r = orc.backward(q, k, v, lam, dO, transport="exchange")
        loss = lambda q_, k_, v_, l_: float(np.sum(dO * orc.forward(q_, k_, v_, l_, want_matrices=False,
                                                                     transport="exchange")["Y"]))
        h = 1e-6
        for name, X in (("dq", q), ("dk", k), ("dv", v)):
            num = np.empty_like(X)
            for idx in np.ndindex(X.shape):
                old = X[idx]
                X[idx] = old + h
                lp = loss(q, k, v, lam)
                X[idx] = old - h
                lm = loss(q, k, v, lam)
                X[idx] = old
                num[idx] = (lp - lm) / (2 * h)
            assert np.allclose(r[name], num, atol=2e-8), f"exchange-only {name} vs FD"
        num_l = (loss(q, k, v, lam + h) - loss(q, k, v, lam - h)) / (2 * h)
        assert abs(r["dlam"] - num_l) < 2e-8, "exchange-only dlam vs FD"
        # the columns of dV add up to the rows of dO weighted by the Exchange mass g_i
        assert np.allclose(r["dv"].sum(0), (g["exch_mass"][:, None] * dO).sum(0), atol=1e-12)


ALL_CHECKS = [
    check_brute_force, check_invariants, check_flash_scan, check_closed_forms,
    check_lambda_limits, check_gradients_fd, check_routes_agree,
    check_gradient_special_cases, check_row_blocking, check_exchange_only,
]
