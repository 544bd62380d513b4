"""fp64 CPU oracle for the causal Full Relation operator (Self-Exchange Relation).

TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
baseline leg may import this module. The product path (the HIP library and its
Python binding) never calls it, and it shares no code with that path.

What it computes: the plain definition of one Relation head, written out in
fp64 with the T x T matrices materialised, following the paper:
  * pairwise evidence  U_ij = p1_i . p2_j / sqrt(d_h)                 (eq. 1)
  * Self map           S_i  = sigmoid(U_ii / tau_S), tau_S = 2        (eq. 2)
  * Exchange map       E_ij = SiLU(U_ij)                              (eq. 2)
  * causal Relation    R_ii = S_i; R_ij = E_ij - lambda log i (j < i);
                       R_ij = -inf (j > i); i is one-based            (eq. 2; App. A.1.1)
  * flow and transport F_i = Softmax(R_i), Y_i = sum_{j<=i} F_ij I~_j (eq. 3)
The derived quantities (Self mass, aggregate Exchange mass g, Exchange
log-normaliser L^E, count-corrected aggregate A, allocation pi) follow
eqs. (5)-(7) / App. A.1.2-A.1.4. The backward pass is computed by two
independent routes from App. A.1.7: through the softmax Jacobian of F, and
through the Self-Exchange factorisation (g, pi, c).

The oracle consumes exactly the values given to the GPU (bf16 inputs are
rounded by the caller and passed here as fp64). Library primitives used as
steps: numpy matmul, scipy.special.expit / softmax / logsumexp.

Conventions where the paper leaves a choice (each is listed with its reason in
the design notes): the log is natural; row 1 has an empty history, so its
L^E and A are -inf, g_1 = 0 and pi_1 = 0; the saved statistic for the
backward pass is M_i = ln Z_i + lambda ln i.

Rows are processed in blocks of ``row_block`` rows purely to bound memory at
long T. Rows of F are independent (each is its own softmax), so the blocking
changes no arithmetic of a row; only the order of the column sums that form
dK and dV changes, at fp64 rounding level.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import expit, logsumexp, softmax

__all__ = ["forward", "backward", "TAU_S"]

TAU_S = 2.0  # Self temperature used in all of the paper's experiments (Sec. 3.1)


def _scale(D: int, scale: float | None) -> float:
    # 1/sqrt(d_h) sits inside U (eq. 1)
    return 1.0 / math.sqrt(D) if scale is None else float(scale)


def _row_block_matrices(q, k, lam, tau_s, s, rows):
    """U, S, E, R for the query rows ``rows`` (zero-based indices) of one head,
    all columns. Returns U_blk [nb, T], S_blk [nb], E_blk [nb, T], R_blk [nb, T].
    """
    T = k.shape[0]
    nb = len(rows)
    U = s * (q[rows] @ k.T)                         # eq. (1)
    S = expit(U[np.arange(nb), rows] / tau_s)       # eq. (2), Self on the diagonal
    E = U * expit(U)                                # eq. (2), SiLU(U) = U sigmoid(U)
    ione = (rows + 1).astype(np.float64)            # one-based count index (App. A.1.1)
    R = np.full_like(U, -np.inf)
    cols = np.arange(T)
    below = cols[None, :] < rows[:, None]           # j < i: historical Exchange entries
    R[below] = (E - lam * np.log(ione)[:, None])[below]
    R[np.arange(nb), rows] = S                      # j = i: Self
    return U, S, E, R


def forward(q, k, v, lam, *, tau_s: float = TAU_S, scale: float | None = None,
            want_matrices: bool = True, row_block: int | None = None, rows=None,
            transport: str = "full") -> dict:
    """Full Relation forward for one head. q, k, v: [T, D] fp64 arrays.

    ``transport="exchange"`` is the exchange-only ablation (App. D, ablation
    definitions): the same F, but Y_i = sum_{j<i} F_ij I~_j, without the Self
    term and without renormalising the historical weights.

    ``rows`` (optional, increasing zero-based indices) restricts the output to
    those query rows; each row of F is its own softmax, so a row's result does
    not depend on which other rows are evaluated.

    Returns a dict with, per evaluated row i: Y [n, D], S, self_mass (F_ii),
    exch_mass (g), LE (L^E, -inf for row 1), A, lnZ, M (= ln Z + lambda ln i);
    and, when ``want_matrices``, the [n, T] rows of U, E, R, F and pi
    (pi_ij = F_ij / g_i for j < i, zero elsewhere and on row 1).
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    T, D = q.shape
    lam = float(lam)
    s = _scale(D, scale)
    rows = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    n = len(rows)
    rb = max(n, 1) if row_block is None else max(1, int(row_block))
    exch_only = _transport(transport)

    Y = np.empty((n, D))
    S = np.empty(n)
    self_mass = np.empty(n)
    g = np.empty(n)
    LE = np.empty(n)
    lnZ = np.empty(n)
    mats = {m: np.empty((n, T)) for m in ("U", "E", "R", "F", "pi")} if want_matrices else None

    for b0 in range(0, n, rb):
        b1 = min(n, b0 + rb)
        rr = rows[b0:b1]
        U, Sb, E, R = _row_block_matrices(q, k, lam, tau_s, s, rr)
        F = softmax(R, axis=1)                       # eq. (3): F_i = Softmax(R_i)
        Ft = F
        if exch_only:                                # transport of historical entries only
            Ft = F.copy()
            Ft[np.arange(b1 - b0), rr] = 0.0
        Y[b0:b1] = Ft @ v                            # eq. (3): Y_i = sum_j F_ij I~_j
        S[b0:b1] = Sb
        diagF = F[np.arange(b1 - b0), rr]
        self_mass[b0:b1] = diagF
        below = np.arange(T)[None, :] < rr[:, None]
        g[b0:b1] = np.where(below, F, 0.0).sum(axis=1)       # g_i = sum_{j<i} F_ij (eq. 6)
        LE[b0:b1] = logsumexp(np.where(below, E, -np.inf), axis=1)  # L^E_i (eq. 5)
        lnZ[b0:b1] = logsumexp(R, axis=1)
        if want_matrices:
            mats["U"][b0:b1] = U
            mats["E"][b0:b1] = E
            mats["R"][b0:b1] = R
            mats["F"][b0:b1] = F
            with np.errstate(invalid="ignore", divide="ignore"):
                pi = np.where(below, F / g[b0:b1, None], 0.0)  # pi_ij = F_ij / g_i (eq. 7)
            mats["pi"][b0:b1] = pi

    ione = (rows + 1).astype(np.float64)
    A = LE - lam * np.log(ione)                      # A_i = L^E_i - lambda log i (eq. 5)
    out = {
        "Y": Y, "S": S, "self_mass": self_mass, "exch_mass": g, "LE": LE, "A": A,
        "lnZ": lnZ, "M": lnZ + lam * np.log(ione), "scale": s, "lam": lam, "tau_s": tau_s,
        "rows": rows,
    }
    if want_matrices:
        out.update(mats)
    return out


def _transport(transport: str) -> bool:
    if transport not in ("full", "exchange"):
        raise ValueError(f"unknown transport {transport!r}")
    return transport == "exchange"


def _silu_grad(U):
    # d SiLU(U) / dU = sigmoid(U) + U sigmoid(U) (1 - sigmoid(U))   (App. A.1.7)
    sg = expit(U)
    return sg + U * sg * (1.0 - sg)


def backward(q, k, v, lam, dout, *, tau_s: float = TAU_S, scale: float | None = None,
             route: str = "softmax", row_block: int | None = None, rows=None,
             transport: str = "full") -> dict:
    """Gradients of sum(dout * Y) for one head.

    Returns dq, dk, dv [T, D], dlam (this head's contribution; lambda is shared
    across heads, so the layer's gradient is the sum over heads) and dS [T]
    (the gradient with respect to the Self logit R_ii = S_i).

    route="softmax": through the softmax Jacobian of F (App. A.1.7, general
        Relation transport): H_ij = G_i . I~_j, dR_ij = F_ij (H_ij - sum_k F_ik H_ik),
        then the role-map derivatives and dlam = -sum_i log i sum_{j<i} dR_ij.
    route="factorised": through g, pi and c_i = G_i . (Ibar_i - I~_i)
        (App. A.1.7, Self-Exchange credit decomposition).

    ``rows`` (softmax route only; increasing zero-based indices) evaluates only
    the contributions of those query rows: dq, dS and dlam for those rows, and
    dk, dv summed over those rows. With rows = {j0, ..., T-1}, dk_j and dv_j are
    complete for every j >= j0, since only rows i >= j reach key j.

    ``transport="exchange"`` (softmax route only): gradients of the
    exchange-only output, where Y_i does not depend on F_ii, so dL/dF_ii = 0
    and I~_i receives nothing from its own row.
    """
    if route == "softmax":
        return _backward_softmax(q, k, v, lam, dout, tau_s, scale, row_block, rows, _transport(transport))
    if rows is not None or _transport(transport):
        raise ValueError("row subsets and exchange-only transport are evaluated by the softmax route")
    if route == "factorised":
        return _backward_factorised(q, k, v, lam, dout, tau_s, scale)
    raise ValueError(f"unknown route {route!r}")


def _backward_softmax(q, k, v, lam, dout, tau_s, scale, row_block, rows, exch_only=False):
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    G = np.asarray(dout, np.float64)
    T, D = q.shape
    lam = float(lam)
    s = _scale(D, scale)
    rows = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    n = len(rows)
    rb = max(n, 1) if row_block is None else max(1, int(row_block))
    dq = np.empty((n, D))
    dk = np.zeros((T, D))
    dv = np.zeros((T, D))
    dS = np.empty(n)
    dlam = 0.0
    for b0 in range(0, n, rb):
        b1 = min(n, b0 + rb)
        rr = rows[b0:b1]
        nb = b1 - b0
        U, Sb, E, R = _row_block_matrices(q, k, lam, tau_s, s, rr)
        F = softmax(R, axis=1)
        Gb = G[rr]
        H = Gb @ v.T                                   # H_ij = G_i . I~_j = dL/dF_ij
        Ft = F
        if exch_only:                                  # F_ii is not transported
            H[np.arange(nb), rr] = 0.0
            Ft = F.copy()
            Ft[np.arange(nb), rr] = 0.0
        Drow = (F * H).sum(axis=1)                     # sum_{k<=i} F_ik H_ik
        dR = F * (H - Drow[:, None])                   # softmax Jacobian (zero where F = 0)
        below = np.arange(T)[None, :] < rr[:, None]
        diag = (np.arange(nb), rr)
        dU = np.where(below, dR * _silu_grad(U), 0.0)  # Exchange entries: dE/dU = SiLU'(U)
        dU[diag] = dR[diag] * Sb * (1.0 - Sb) / tau_s  # Self entry: dS/dU_ii = S(1-S)/tau_S
        dq[b0:b1] = s * (dU @ k)                       # grad P1 = grad_U P2 / sqrt(d_h)
        dk += s * (dU.T @ q[rr])                       # grad P2 = grad_U^T P1 / sqrt(d_h)
        dv += Ft.T @ Gb                                # dL/dI~_j = sum_i F_ij G_i (transported entries)
        dS[b0:b1] = dR[diag]
        ione = (rr + 1).astype(np.float64)
        dlam += float(-(np.log(ione) * np.where(below, dR, 0.0).sum(axis=1)).sum())
    return {"dq": dq, "dk": dk, "dv": dv, "dlam": dlam, "dS": dS, "rows": rows}


def _backward_factorised(q, k, v, lam, dout, tau_s, scale):
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    G = np.asarray(dout, np.float64)
    T, D = q.shape
    f = forward(q, k, v, lam, tau_s=tau_s, scale=scale, want_matrices=True)
    s = f["scale"]
    U, S, g, pi = f["U"], f["S"], f["exch_mass"], f["pi"]
    # Exchange aggregate Ibar_i = sum_{j<i} pi_ij I~_j (eq. 8); row 1 has none and
    # enters only through g_1 = 0, so it is left at zero.
    Ibar = pi @ v
    Delta = Ibar - v                                  # Delta_i = Ibar_i - I~_i
    c = (G * Delta).sum(axis=1)                       # c_i = G_i . Delta_i
    below = np.tril(np.ones((T, T), dtype=bool), k=-1)
    # dL/dE_ij = g_i pi_ij [ (1-g_i) c_i + G_i . (I~_j - Ibar_i) ]
    GI = G @ v.T                                      # G_i . I~_j
    GIbar = (G * Ibar).sum(axis=1)                    # G_i . Ibar_i
    dE = np.where(below, g[:, None] * pi * ((1.0 - g) * c)[:, None]
                  + g[:, None] * pi * (GI - GIbar[:, None]), 0.0)
    dS = -g * (1.0 - g) * c                           # dL/dS_i = -g_i (1 - g_i) c_i
    dU = np.where(below, dE * _silu_grad(U), 0.0)
    dU[np.diag_indices(T)] = dS * S * (1.0 - S) / tau_s
    dq = s * (dU @ k)
    dk = s * (dU.T @ q)
    # dL/dI~_j = (1 - g_j) G_j + sum_{i>j} g_i pi_ij G_i
    dv = (1.0 - g)[:, None] * G + (g[:, None] * pi).T @ G
    ione = np.arange(1, T + 1, dtype=np.float64)
    # dL/dlambda = -sum_{i>1} g_i (1 - g_i) c_i log i
    dlam = float(-(g * (1.0 - g) * c * np.log(ione))[1:].sum())
    return {"dq": dq, "dk": dk, "dv": dv, "dlam": dlam, "dS": dS}


def forward_batched(q, k, v, lam, **kw) -> dict:
    """Apply ``forward`` to every (b, h) head of [B, H, T, D] arrays (heads are
    independent, Sec. 3.2 / App. A.2.1). Row quantities come back as [B, H, T]."""
    B, H, T, D = q.shape
    keys = ("Y", "S", "self_mass", "exch_mass", "LE", "A", "lnZ", "M")
    out = {"Y": np.empty((B, H, T, D))}
    for key in keys[1:]:
        out[key] = np.empty((B, H, T))
    kw = dict(kw)
    kw.setdefault("want_matrices", False)
    for b in range(B):
        for h in range(H):
            f = forward(q[b, h], k[b, h], v[b, h], lam, **kw)
            for key in keys:
                out[key][b, h] = f[key]
    return out


def backward_batched(q, k, v, lam, dout, **kw) -> dict:
    """Apply ``backward`` to every head; dlam is summed over heads because
    lambda is one scalar per layer shared by all heads (App. A.1.1)."""
    B, H, T, D = q.shape
    out = {n: np.empty((B, H, T, D)) for n in ("dq", "dk", "dv")}
    out["dS"] = np.empty((B, H, T))
    dlam = 0.0
    for b in range(B):
        for h in range(H):
            r = backward(q[b, h], k[b, h], v[b, h], lam, dout[b, h], **kw)
            for n in ("dq", "dk", "dv", "dS"):
                out[n][b, h] = r[n]
            dlam += r["dlam"]
    out["dlam"] = dlam
    return out
