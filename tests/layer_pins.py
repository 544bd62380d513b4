"""Checks that pin the layer oracle (RoPE, Givens mixing, their backward) to
facts fixed by the paper and by mathematics, independently of its own code.

Each ``check_*`` takes the layer-oracle module under test and raises
AssertionError on a mismatch. ``test_layer_oracle.py`` runs them on the real
module and on copies with planted mistakes.
"""
from __future__ import annotations

import math
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------------------
# RoPE
# ---------------------------------------------------------------------------
def check_rope_d4_closed_form(lo):
    """Head width 4: the two channel pairs turn at 1 and base^(-1/2) radians per
    position, i.e. 1 and 0.01 for base 10^4, 1 and 0.1 for base 100 (worked by
    hand from the rotary definition with the full-width pairing (d, d + 2))."""
    T = 9
    x = np.tile(np.array([1.0, 2.0, 3.0, 4.0]), (T, 1))
    for base, slow in ((1.0e4, 0.01), (100.0, 0.1)):
        y = lo.rope(x, base)
        for t in range(T):
            a, b = t * 1.0, t * slow
            want = [1 * math.cos(a) - 3 * math.sin(a), 2 * math.cos(b) - 4 * math.sin(b),
                    1 * math.sin(a) + 3 * math.cos(a), 2 * math.sin(b) + 4 * math.cos(b)]
            assert np.allclose(y[t], want, atol=1e-14), f"rope d=4 base={base} t={t}"


def check_rope_invariants(lo):
    rng = _rng(1)
    T, D = 40, 16
    x = rng.standard_normal((2, 3, T, D))
    y = lo.rope(x)
    # a rotation: norms kept, position 0 untouched
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), atol=1e-12), "norm"
    assert np.array_equal(y[..., 0, :], x[..., 0, :]), "position 0"
    # relative position: the same q and k at every position give a score that
    # depends only on the offset m - n (Toeplitz)
    qv, kv = rng.standard_normal(D), rng.standard_normal(D)
    Q, K = lo.rope(np.tile(qv, (T, 1))), lo.rope(np.tile(kv, (T, 1)))
    S = Q @ K.T
    for off in (-7, 0, 3, 11):
        dg = np.diagonal(S, offset=off)
        assert np.allclose(dg, dg[0], atol=1e-11), f"score depends on absolute position (offset {off})"
    # and it does depend on the offset
    assert not np.allclose(np.diagonal(S, 1)[0], np.diagonal(S, 5)[0])


def check_rope_transpose(lo):
    rng = _rng(2)
    x, g = rng.standard_normal((2, 2, 33, 12)), rng.standard_normal((2, 2, 33, 12))
    assert np.allclose(lo.rope_transpose(lo.rope(x)), x, atol=1e-12), "inverse"
    # adjoint: <rope(x), g> = <x, rope^T(g)>
    assert abs(np.sum(lo.rope(x) * g) - np.sum(x * lo.rope_transpose(g))) < 1e-10, "adjoint"


# ---------------------------------------------------------------------------
# Givens mixing
# ---------------------------------------------------------------------------
def check_givens_pairings(lo):
    """The two pairings for H = 8 as the paper lists them (one-based)."""
    rows = {}
    for ln in open(os.path.join(GOLDEN, "givens_pairings_h8.txt")):
        if ln.strip() and not ln.startswith("#"):
            name, *idx = ln.split()
            idx = [int(t) - 1 for t in idx]
            rows[name] = list(zip(idx[0::2], idx[1::2]))
    for name in ("A", "B"):
        assert [tuple(p) for p in lo.givens_pairs(8, name)] == rows[name], f"pairing {name}"
    # every head sits in exactly one pair of each pairing
    for H in (2, 4, 12):
        for name in ("A", "B"):
            heads = sorted(h for p in lo.givens_pairs(H, name) for h in p)
            assert heads == list(range(H)), f"pairing {name} H={H}"


def check_givens_closed_forms(lo):
    rng = _rng(3)
    B, H, T, D = 2, 4, 5, 3
    I = rng.standard_normal((B, H, T, D))
    for pairing in ("A", "B"):
        pairs = lo.givens_pairs(H, pairing)
        assert np.allclose(lo.givens(I, np.zeros(H // 2), pairing), I, atol=0), "theta 0"
        # a quarter turn: I~a = -Ib, I~b = Ia (eq. 4 with cos = 0, sin = 1)
        Q = lo.givens(I, np.full(H // 2, math.pi / 2), pairing)
        for a, b in pairs:
            assert np.allclose(Q[:, a], -I[:, b], atol=1e-15) and np.allclose(Q[:, b], I[:, a], atol=1e-15)
        # orthogonal per pair (App. A.2.2): squared norms of a pair are kept
        th = rng.uniform(-3, 3, H // 2)
        M = lo.givens(I, th, pairing)
        for a, b in pairs:
            n0 = np.sum(I[:, a] ** 2) + np.sum(I[:, b] ** 2)
            n1 = np.sum(M[:, a] ** 2) + np.sum(M[:, b] ** 2)
            assert abs(n0 - n1) < 1e-12, "pair norm"
        # a pair's angle moves only that pair's heads
        th2 = th.copy()
        th2[0] += 0.3
        M2 = lo.givens(I, th2, pairing)
        untouched = [h for h in range(H) if h not in pairs[0]]
        assert np.array_equal(M2[:, untouched], M[:, untouched]), "other pairs move"


def check_givens_grad_fd(lo):
    rng = _rng(4)
    B, H, T, D = 2, 4, 3, 2
    I = rng.standard_normal((B, H, T, D))
    G = rng.standard_normal((B, H, T, D))
    for pairing in ("A", "B"):
        th = rng.uniform(-2, 2, H // 2)
        dI, dth = lo.givens_backward(G, I, th, pairing)
        f = lambda I_, th_: float(np.sum(G * lo.givens(I_, th_, pairing)))
        h = 1e-6
        for p in range(H // 2):
            e = np.zeros(H // 2)
            e[p] = h
            fd = (f(I, th + e) - f(I, th - e)) / (2 * h)
            assert abs(fd - dth[p]) < 1e-7 * max(1.0, abs(fd)), f"dtheta[{p}] {pairing}"
        for idx in [(0, 0, 0, 0), (1, 3, 2, 1), (0, 1, 1, 0), (1, 2, 0, 1)]:
            E = np.zeros_like(I)
            E[idx] = h
            fd = (f(I + E, th) - f(I - E, th)) / (2 * h)
            assert abs(fd - dI[idx]) < 1e-7 * max(1.0, abs(fd)), f"dI{idx} {pairing}"


# ---------------------------------------------------------------------------
# The layer: composition and its gradients
# ---------------------------------------------------------------------------
def check_layer_off_is_operator(lo):
    rng = _rng(5)
    q, k, v = (rng.standard_normal((1, 2, 11, 4)) for _ in range(3))
    f = lo.layer_forward(q, k, v, 0.3, None, None, rope_base=0.0)
    g = oracle.forward_batched(q, k, v, 0.3)
    assert np.array_equal(f["Y"], g["Y"]), "no RoPE, no mixing"


def check_layer_grad_fd(lo):
    """Central differences of sum(dO * Y) through RoPE, Givens and the operator."""
    rng = _rng(6)
    B, H, T, D = 1, 4, 7, 4
    q, k, v, dO = (rng.standard_normal((B, H, T, D)) for _ in range(4))
    th = rng.uniform(-1, 1, H // 2)
    lam = 0.4
    for pairing, base in (("A", 1.0e4), ("B", 10.0)):
        r = lo.layer_backward(q, k, v, lam, dO, th, pairing, base)
        L = lambda q_, k_, v_, lam_, th_: float(np.sum(dO * lo.layer_forward(
            q_, k_, v_, lam_, th_, pairing, base)["Y"]))
        h = 1e-6
        for name, arr, grad in (("q", q, r["dq"]), ("k", k, r["dk"]), ("v", v, r["dv"])):
            for idx in [(0, 0, 3, 0), (0, 1, 6, 3), (0, 3, 5, 2), (0, 2, 1, 1)]:
                E = np.zeros_like(arr)
                E[idx] = h
                args_p = {"q": q, "k": k, "v": v}
                args_m = dict(args_p)
                args_p[name], args_m[name] = arr + E, arr - E
                fd = (L(args_p["q"], args_p["k"], args_p["v"], lam, th)
                      - L(args_m["q"], args_m["k"], args_m["v"], lam, th)) / (2 * h)
                assert abs(fd - grad[idx]) < 1e-6 * max(1.0, abs(fd)), f"d{name}{idx} {pairing}"
        for p in range(H // 2):
            e = np.zeros(H // 2)
            e[p] = h
            fd = (L(q, k, v, lam, th + e) - L(q, k, v, lam, th - e)) / (2 * h)
            assert abs(fd - r["dtheta"][p]) < 1e-6 * max(1.0, abs(fd)), f"dtheta[{p}] {pairing}"
        fd = (L(q, k, v, lam + h, th) - L(q, k, v, lam - h, th)) / (2 * h)
        assert abs(fd - r["dlam"]) < 1e-6 * max(1.0, abs(fd)), f"dlam {pairing}"


ALL_CHECKS = [
    check_rope_d4_closed_form,
    check_rope_invariants,
    check_rope_transpose,
    check_givens_pairings,
    check_givens_closed_forms,
    check_givens_grad_fd,
    check_layer_off_is_operator,
    check_layer_grad_fd,
]
