"""Shared helpers for the GPU parity tests: move seeded inputs to the device,
run the oracle on the same (rounded) values, and compare."""
from __future__ import annotations

import math
import sys

import numpy as np
import torch

import oracle

TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16}

# Bars: fp32 max-abs <= 1e-4; bf16 relative l2 <= 2e-2 (outputs and gradients).
F32_MAX_ABS = 1e-4
BF16_REL_L2 = 2e-2


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def to_device(arr: np.ndarray, dtype: str):
    """fp64 numpy -> device tensor of ``dtype`` and the fp64 copy of exactly the
    values stored on the device (the oracle's input)."""
    t = torch.from_numpy(np.ascontiguousarray(arr)).to(TORCH_DT[dtype])
    rounded = t.to(torch.float64).numpy()
    return t.cuda(), rounded


def lam_value(lam: float) -> float:
    # lambda is stored in fp32 on the device (App. A.1.1); the oracle uses that value
    return float(np.float32(lam))


def rel_l2(x: np.ndarray, ref: np.ndarray) -> float:
    den = float(np.linalg.norm(ref.ravel()))
    num = float(np.linalg.norm((x - ref).ravel()))
    return num / den if den > 0 else num


def max_abs(x: np.ndarray, ref: np.ndarray, finite_only: bool = False) -> float:
    d = np.abs(x - ref)
    if finite_only:
        d = d[np.isfinite(ref)]
    return float(d.max()) if d.size else 0.0


def assert_close(name: str, x, ref, dtype: str) -> None:
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert x.shape == ref.shape, f"{name}: shape {x.shape} vs {ref.shape}"
    assert np.all(np.isfinite(x) == np.isfinite(ref)), f"{name}: non-finite pattern differs"
    fin = np.isfinite(ref)
    if not np.array_equal(x[~fin], ref[~fin]):
        raise AssertionError(f"{name}: infinite entries differ")
    if dtype == "f32":
        err = max_abs(x[fin], ref[fin])
        log(f"  {name}: max-abs {err:.3e} (bar {F32_MAX_ABS:g})")
        assert err <= F32_MAX_ABS, f"{name}: max-abs {err:.3e} > {F32_MAX_ABS:g}"
    else:
        err = rel_l2(x[fin], ref[fin])
        log(f"  {name}: rel-l2 {err:.3e} (bar {BF16_REL_L2:g})")
        assert err <= BF16_REL_L2, f"{name}: rel-l2 {err:.3e} > {BF16_REL_L2:g}"


def assert_scalar_close(name: str, x: float, ref: float, terms, dtype: str) -> None:
    """A scalar that is a signed sum of many per-row terms (dlambda, dtheta),
    given with the array of its reference terms. Such a sum can cancel, so its
    error is held to the bar relative to the larger of |ref| and the l2 norm of
    the term vector: |x - ref| <= bar * max(|ref|, ||terms||_2). Without
    cancellation this is the relative bar; with it, it is the error that term
    errors within the relative-l2 bar give when they are uncorrelated. fp32:
    max-abs against the larger of the fp32 bar and 1e-5 of sum |terms|."""
    t = np.abs(np.asarray(terms, dtype=np.float64)).ravel()
    terms_abs, terms_l2 = float(t.sum()), float(np.sqrt(np.sum(t * t)))
    bar = F32_MAX_ABS if dtype == "f32" else BF16_REL_L2
    err = abs(x - ref)
    rel = err / abs(ref) if ref != 0 else math.inf
    rel_l2t = err / terms_l2 if terms_l2 > 0 else err
    log(f"  {name}: gpu {x:.6e} ref {ref:.6e} rel {rel:.3e} rel-to-||terms||2 {rel_l2t:.3e}")
    if dtype == "f32":
        assert err <= max(F32_MAX_ABS, 1e-5 * terms_abs), f"{name}: abs err {err:.3e}"
    else:
        ok = err == 0.0 or err <= bar * max(abs(ref), terms_l2) or (terms_l2 == 0.0 and err <= 1e-6)
        assert ok, f"{name}: rel {rel:.3e}, rel-to-||terms||2 {rel_l2t:.3e}"


def oracle_heads(qr, kr, vr, lam, heads, dout=None, row_block=None):
    """Oracle forward (and backward if ``dout``) on the listed (b, h) heads."""
    res = []
    for (b, h) in heads:
        f = oracle.forward(qr[b, h], kr[b, h], vr[b, h], lam, want_matrices=False, row_block=row_block)
        r = None
        if dout is not None:
            r = oracle.backward(qr[b, h], kr[b, h], vr[b, h], lam, dout[b, h], row_block=row_block)
        res.append((f, r))
    return res


def sample_heads(B: int, H: int, k: int = 3):
    cand = [(0, 0), (B - 1, H - 1), (B // 2, H // 2), (0, H - 1), (B - 1, 0)]
    out = []
    for c in cand:
        if c not in out:
            out.append(c)
    return out[:k]


# dq of the one-kernel backward sums per-workgroup partials with fp32 atomics in
# whatever order they arrive: two runs agree to fp32 rounding, and after the
# bf16 rounding of the output a few elements may differ by one unit in the last
# place.
ATOMIC_ORDER_REL_L2 = 1e-3


def assert_order_close(name: str, x, ref) -> None:
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = rel_l2(x, ref)
    log(f"  {name}: rel-l2 {err:.3e} between runs (bar {ATOMIC_ORDER_REL_L2:g})")
    assert err <= ATOMIC_ORDER_REL_L2, f"{name}: rel-l2 {err:.3e}"
