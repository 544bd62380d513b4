"""fp64 CPU oracle for the steps around one Relation layer's operator: RoPE on
the two relation projections, Givens head-pair mixing of the information
state, and the backward pass through both.

TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
baseline leg may import this module. The product path never calls it, and it
shares no code with that path.

What it computes, following the paper:
  * RoPE (Sec. 3.1 and App. B, position encoding): the head-wise P1 and P2
    are rotated before pairwise evidence is formed; the information
    projection is not. The rotation spans the full head width d_h with base
    10^4.
  * Givens mixing (eq. 4; App. A.2.2-A.2.3): for each head pair (a, b) of
    the layer's pairing, I~(a) = cos t I(a) - sin t I(b) and
    I~(b) = sin t I(a) + cos t I(b), one fp32 angle t per pair, shared by
    every channel and position. Pairing A is (1,2), (3,4), ..., (H-1,H);
    pairing B is (2,3), (4,5), ..., (H,1) (one-based heads).
  * The operator itself on (RoPE(P1), RoPE(P2), I~) is relation_oracle.

Readings where the paper leaves a choice (listed in the design notes):
  * RoPE rotates channel d with channel d + d_h/2 (the "rotate half" pairing)
    by the angle t * base^(-2d/d_h), d = 0 .. d_h/2 - 1, with t the
    zero-based position of the token in its sequence.
  * A head width the kernels do not tile natively is handled by padding with
    zero channels; the oracle works at the true width d_h, and 1/sqrt(d_h)
    uses the true width.
  * The Givens angles are shared by the whole batch, so their gradient sums
    over batch, position and channel.
"""
from __future__ import annotations

import numpy as np

from .relation_oracle import TAU_S, backward_batched, forward_batched

__all__ = ["rope", "rope_transpose", "givens_pairs", "givens", "givens_backward",
           "layer_forward", "layer_backward", "ROPE_BASE"]

ROPE_BASE = 1.0e4  # App. B: base 10^4, no positional scaling


def _rope_cos_sin(T: int, D: int, base: float):
    if D % 2:
        raise ValueError("RoPE needs an even head width")
    half = D // 2
    freq = base ** (-2.0 * np.arange(half) / D)          # one frequency per channel pair
    ang = np.arange(T, dtype=np.float64)[:, None] * freq[None, :]  # [T, D/2]
    return np.cos(ang), np.sin(ang)


def rope(x, base: float = ROPE_BASE):
    """Rotate the last axis of x [..., T, D]: channel d with channel d + D/2."""
    T, D = x.shape[-2], x.shape[-1]
    c, s = _rope_cos_sin(T, D, base)
    x1, x2 = x[..., : D // 2], x[..., D // 2:]
    return np.concatenate([x1 * c - x2 * s, x1 * s + x2 * c], axis=-1)


def rope_transpose(g, base: float = ROPE_BASE):
    """The transposed (inverse) rotation: the gradient with respect to the
    unrotated projection, given the gradient with respect to the rotated one."""
    T, D = g.shape[-2], g.shape[-1]
    c, s = _rope_cos_sin(T, D, base)
    g1, g2 = g[..., : D // 2], g[..., D // 2:]
    return np.concatenate([g1 * c + g2 * s, -g1 * s + g2 * c], axis=-1)


def givens_pairs(H: int, pairing: str):
    """Zero-based (a, b) head pairs of pairing "A" or "B" (App. A.2.3)."""
    if H % 2:
        raise ValueError("Givens mixing pairs heads: H must be even")
    if pairing == "A":
        return [(2 * p, 2 * p + 1) for p in range(H // 2)]
    if pairing == "B":
        return [(2 * p + 1, (2 * p + 2) % H) for p in range(H // 2)]
    raise ValueError(f"unknown pairing {pairing!r}")


def givens(I, theta, pairing: str):
    """I~ from I [B, H, T, D] and one angle per pair (eq. 4)."""
    H = I.shape[1]
    out = np.array(I, dtype=np.float64, copy=True)
    for p, (a, b) in enumerate(givens_pairs(H, pairing)):
        c, s = np.cos(theta[p]), np.sin(theta[p])
        out[:, a] = c * I[:, a] - s * I[:, b]
        out[:, b] = s * I[:, a] + c * I[:, b]
    return out


def givens_backward(dIt, I, theta, pairing: str):
    """Gradients with respect to I and the angles, given dL/dI~."""
    H = I.shape[1]
    dI = np.array(dIt, dtype=np.float64, copy=True)
    dth = np.zeros(len(theta))
    for p, (a, b) in enumerate(givens_pairs(H, pairing)):
        c, s = np.cos(theta[p]), np.sin(theta[p])
        dI[:, a] = c * dIt[:, a] + s * dIt[:, b]       # G^T applied to (dI~a, dI~b)
        dI[:, b] = -s * dIt[:, a] + c * dIt[:, b]
        # d I~a / d t = -s Ia - c Ib ;  d I~b / d t = c Ia - s Ib
        dth[p] = float(np.sum(dIt[:, a] * (-s * I[:, a] - c * I[:, b]))
                       + np.sum(dIt[:, b] * (c * I[:, a] - s * I[:, b])))
    return dI, dth


def _prepare(q, k, v, theta, pairing, rope_base):
    qr = rope(q, rope_base) if rope_base else np.asarray(q, dtype=np.float64)
    kr = rope(k, rope_base) if rope_base else np.asarray(k, dtype=np.float64)
    vt = givens(v, theta, pairing) if pairing else np.asarray(v, dtype=np.float64)
    return qr, kr, vt


def layer_forward(q, k, v, lam, theta=None, pairing=None, rope_base: float = ROPE_BASE, *,
                  tau_s: float = TAU_S, scale=None, **kw):
    """Y of the layer's operator for [B, H, T, D] projections: RoPE on q and k
    (rope_base 0 turns it off), Givens mixing of v (pairing None turns it off),
    then the causal Full Relation per head. Also returns the prepared operands."""
    qr, kr, vt = _prepare(q, k, v, theta, pairing, rope_base)
    f = forward_batched(qr, kr, vt, lam, tau_s=tau_s, scale=scale, **kw)
    f.update({"qr": qr, "kr": kr, "vt": vt})
    return f


def layer_backward(q, k, v, lam, dout, theta=None, pairing=None, rope_base: float = ROPE_BASE, *,
                   tau_s: float = TAU_S, scale=None, **kw):
    """Gradients of sum(dout * Y) with respect to q, k, v, lambda and the angles."""
    qr, kr, vt = _prepare(q, k, v, theta, pairing, rope_base)
    r = backward_batched(qr, kr, vt, lam, dout, tau_s=tau_s, scale=scale, **kw)
    dq = rope_transpose(r["dq"], rope_base) if rope_base else r["dq"]
    dk = rope_transpose(r["dk"], rope_base) if rope_base else r["dk"]
    if pairing:
        dv, dth = givens_backward(r["dv"], v, theta, pairing)
    else:
        dv, dth = r["dv"], None
    return {"dq": dq, "dk": dk, "dv": dv, "dlam": r["dlam"], "dtheta": dth, "dS": r["dS"],
            "dq_rot": r["dq"], "dk_rot": r["dk"], "dvt": r["dv"]}
