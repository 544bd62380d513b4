"""fp64 CPU oracle for Linear Relation (Sec. 5.2, App. A.4): Self kept explicit,
Exchange carried by a recurrent relational state with channel-wise retention.

TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
baseline leg may import this module. The product path never calls it, and it
shares no code with that path.

One head, tokens t = 1..T, inputs after RoPE (App. B):
  S_t   = sigmoid(p1_t . p2_t / (tau_S sqrt(d_h)))             Self
  ^p1_t = p1_t / |p1_t|,  ^p2_t = p2_t / |p2_t|                 relation coordinates
  alpha_t = exp(g_t) in (0, 1]^{d_h}                             retention
  C_t^- = Diag(alpha_t) C_{t-1},  C_0 = 0                        (read state)
  E_t   = S_t (C_t^-)^T ^p1_t                                    Ask Others
  Y_t   = I~_t + E_t                                             Answer
  C_t   = C_t^- + S_t ^p2_t I~_t^T                               Become Others
The oracle runs this recurrence token by token (``forward``) and its exact
adjoint token by token in reverse (``backward``).

The retention gate of eq. 15 (``kda_gate``) maps the pre-activation r_t and
the per-channel parameters A_log, dt_bias to g_t = log alpha_t; ``forward``
and ``backward`` take g_t itself, and ``kda_gate_backward`` carries dg on to
r, A_log and dt_bias.

Readings where the paper leaves a choice (listed in the design notes):
  * A_log and dt_bias hold one value per channel of the head (the width of
    r_t and alpha_t), shared by every token and batch entry.
  * The state's rows are indexed by the relation channel (the ^p1 / ^p2 side)
    and its columns by the information channel, as written in App. A.4.
  * The scale inside S_t is 1/sqrt(d_h) unless given.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import expit

__all__ = ["forward", "backward", "forward_unrolled", "kda_gate", "kda_gate_backward", "TAU_S"]

TAU_S = 2.0


def _scale(D, scale):
    return 1.0 / math.sqrt(D) if scale is None else float(scale)


def forward(p1, p2, v, g, *, tau_s: float = TAU_S, scale=None, C0=None) -> dict:
    """Y [T, D], S [T] and the final state C [D, D] of one head ([T, D] fp64
    arrays; g is the log-retention). ``C0`` is the state before token 1."""
    p1, p2, v, g = (np.asarray(x, np.float64) for x in (p1, p2, v, g))
    T, D = p1.shape
    s = _scale(D, scale)
    C = np.zeros((D, D)) if C0 is None else np.array(C0, np.float64)
    Y = np.empty((T, D))
    S = np.empty(T)
    for t in range(T):
        S[t] = expit(s * float(p1[t] @ p2[t]) / tau_s)        # Ask Self
        h1 = p1[t] / np.linalg.norm(p1[t])
        h2 = p2[t] / np.linalg.norm(p2[t])
        Cm = np.exp(g[t])[:, None] * C                        # Diag(alpha_t) C_{t-1}
        Y[t] = v[t] + S[t] * (Cm.T @ h1)                      # Answer = I~ + Ask Others
        C = Cm + S[t] * np.outer(h2, v[t])                    # Become Others
    return {"Y": Y, "S": S, "C": C}


def forward_unrolled(p1, p2, v, g, *, tau_s: float = TAU_S, scale=None) -> np.ndarray:
    """Y from the unrolled sum of App. A.4: E_t = sum_{j<t} S_t S_j
    [^p2_j^T (prod_{u=j+1..t} D_u) ^p1_t] I~_j, with the retention products
    taken channel by channel."""
    p1, p2, v, g = (np.asarray(x, np.float64) for x in (p1, p2, v, g))
    T, D = p1.shape
    s = _scale(D, scale)
    S = expit(s * np.einsum("td,td->t", p1, p2) / tau_s)
    h1 = p1 / np.linalg.norm(p1, axis=1, keepdims=True)
    h2 = p2 / np.linalg.norm(p2, axis=1, keepdims=True)
    Y = v.copy()
    for t in range(T):
        for j in range(t):
            prod = np.exp(g[j + 1:t + 1].sum(axis=0))           # prod_{u=j+1}^{t} alpha_u
            Y[t] += S[t] * S[j] * float(np.sum(h2[j] * prod * h1[t])) * v[j]
    return Y


def backward(p1, p2, v, g, dY, *, tau_s: float = TAU_S, scale=None) -> dict:
    """Gradients of sum(dY * Y) with respect to p1, p2, v and g, by running
    the recurrence's adjoint from the last token to the first."""
    p1, p2, v, g, dY = (np.asarray(x, np.float64) for x in (p1, p2, v, g, dY))
    T, D = p1.shape
    s = _scale(D, scale)
    # forward pass, keeping what the adjoint reads
    Cs = np.zeros((T + 1, D, D))                                # Cs[t] = C_{t-1} before token t
    S = np.empty(T)
    n1, n2 = np.linalg.norm(p1, axis=1), np.linalg.norm(p2, axis=1)
    h1, h2 = p1 / n1[:, None], p2 / n2[:, None]
    C = np.zeros((D, D))
    for t in range(T):
        Cs[t] = C
        S[t] = expit(s * float(p1[t] @ p2[t]) / tau_s)
        Cm = np.exp(g[t])[:, None] * C
        C = Cm + S[t] * np.outer(h2[t], v[t])
    dp1, dp2, dv, dg = (np.zeros((T, D)) for _ in range(4))
    dC = np.zeros((D, D))                                       # dL/dC_t after token t
    for t in range(T - 1, -1, -1):
        a = np.exp(g[t])
        Cm = a[:, None] * Cs[t]
        # C_t = Cm + S_t ^p2_t I~_t^T
        dCm = dC.copy()
        dS = float(np.sum(dC * np.outer(h2[t], v[t])))
        dh2 = S[t] * (dC @ v[t])
        dv[t] = S[t] * (dC.T @ h2[t]) + dY[t]                   # the write, and Y_t = I~_t + E_t
        # E_t = S_t Cm^T ^p1_t
        dS += float(dY[t] @ (Cm.T @ h1[t]))
        dCm += S[t] * np.outer(h1[t], dY[t])
        dh1 = S[t] * (Cm @ dY[t])
        # Cm = Diag(exp g_t) C_{t-1}
        dg[t] = a * np.sum(dCm * Cs[t], axis=1)
        dC = a[:, None] * dCm
        # S_t = sigmoid(s p1 . p2 / tau_S)
        dU = dS * S[t] * (1.0 - S[t]) * s / tau_s
        dp1[t] += dU * p2[t]
        dp2[t] += dU * p1[t]
        # ^p = p / |p|
        dp1[t] += (dh1 - h1[t] * float(h1[t] @ dh1)) / n1[t]
        dp2[t] += (dh2 - h2[t] * float(h2[t] @ dh2)) / n2[t]
    return {"dp1": dp1, "dp2": dp2, "dv": dv, "dg": dg}


def kda_gate(r, a_log, dt_bias) -> np.ndarray:
    """Log-retention of eq. 15: g_t = -exp(A_log) * softplus(r_t + dt_bias)
    elementwise, r of shape [..., D] and A_log, dt_bias of shape [D]. Since
    exp > 0 and softplus > 0, g < 0 and alpha = exp(g) lies in (0, 1]."""
    r, a_log, dt_bias = (np.asarray(x, np.float64) for x in (r, a_log, dt_bias))
    softplus = np.logaddexp(0.0, r + dt_bias)                  # log(1 + e^x)
    return -np.exp(a_log) * softplus


def kda_gate_backward(r, a_log, dt_bias, dg) -> dict:
    """Gradients through eq. 15 given dg = dL/dg_t (shape of r): softplus' is
    the logistic sigmoid, so dr = dg * (-exp(A_log) sigmoid(r + dt_bias));
    dt_bias enters as r does, so d dt_bias is dr summed over every axis but
    the channel; and d g / d A_log = g, so d A_log sums dg * g the same way."""
    r, a_log, dt_bias, dg = (np.asarray(x, np.float64) for x in (r, a_log, dt_bias, dg))
    dr = dg * (-np.exp(a_log) * expit(r + dt_bias))
    lead = tuple(range(r.ndim - 1))
    return {"dr": dr, "da_log": np.sum(dg * kda_gate(r, a_log, dt_bias), axis=lead),
            "ddt_bias": np.sum(dr, axis=lead)}
