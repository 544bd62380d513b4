"""Python binding of librelation.so (ctypes). Argument marshalling only: every
step of the operator runs in the library's HIP kernels; torch provides device
memory and the current stream.

Functions carry the C-ABI names (relation_fwd, relation_bwd,
relation_bwd_noalloc, relation_fwd_materialized, relation_bwd_materialized,
relation_exchange_allocation, relation_layer_fwd, relation_layer_bwd,
relation_decode, relation_decode_states, relation_decode_merge, ...). ``relation`` is the differentiable wrapper
(torch.autograd.Function) over relation_fwd / relation_bwd.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librelation.so")

REL_OK, REL_ERR_INVALID_ARG, REL_ERR_UNSUPPORTED, REL_ERR_WORKSPACE, REL_ERR_HIP = 0, -1, -2, -3, -4
REL_F32, REL_BF16 = 0, 1
TAU_S = 2.0


class RelProblem(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int64), ("H", ctypes.c_int64), ("T", ctypes.c_int64), ("D", ctypes.c_int64),
        ("dtype", ctypes.c_int32), ("causal", ctypes.c_int32),
        ("tau_s", ctypes.c_float), ("scale", ctypes.c_float),
        ("stride_b", ctypes.c_int64), ("stride_h", ctypes.c_int64), ("stride_t", ctypes.c_int64),
    ]


class RelLayerOpts(ctypes.Structure):
    _fields_ = [("rope_base", ctypes.c_double), ("givens", ctypes.c_int32), ("transport", ctypes.c_int32)]


REL_GIVENS = {None: 0, "A": 1, "B": 2}
REL_TRANSPORT = {"full": 0, "exchange": 1}
ROPE_BASE = 1.0e4

_P = ctypes.c_void_p
_PP = ctypes.POINTER(RelProblem)
_PO = ctypes.POINTER(RelLayerOpts)
_SIGS = {
    "relation_fwd": (ctypes.c_int, [ctypes.POINTER(RelProblem), _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "relation_exchange_allocation": (ctypes.c_int, [ctypes.POINTER(RelProblem), _P, _P, _P, _P, _P]),
    "relation_bwd_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(RelProblem)]),
    "relation_bwd": (ctypes.c_int, [ctypes.POINTER(RelProblem), _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                    _P, _P, _P, ctypes.c_size_t, _P]),
    "relation_bwd_deterministic": (ctypes.c_int, [ctypes.POINTER(RelProblem), _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                                  _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "relation_bwd_noalloc_max_scratch_bytes": (ctypes.c_size_t, []),
    "relation_bwd_noalloc": (ctypes.c_int, [ctypes.POINTER(RelProblem), _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                            _P, _P, _P, _P]),
    "relation_fwd_materialized_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(RelProblem)]),
    "relation_fwd_materialized": (ctypes.c_int, [ctypes.POINTER(RelProblem), _P, _P, _P, _P, _P, _P, _P,
                                                 _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "relation_bwd_materialized_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(RelProblem)]),
    "relation_bwd_materialized": (ctypes.c_int, [ctypes.POINTER(RelProblem), _P, _P, _P, _P, _P, _P, _P, _P,
                                                 _P, _P, ctypes.c_size_t, _P]),
    "relation_layer_saved_bytes": (ctypes.c_size_t, [_PP, _PO]),
    "relation_layer_fwd_workspace_bytes": (ctypes.c_size_t, [_PP, _PO]),
    "relation_layer_fwd": (ctypes.c_int, [_PP, _PO, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P,
                                          ctypes.c_size_t, _P]),
    "relation_layer_bwd_workspace_bytes": (ctypes.c_size_t, [_PP, _PO]),
    "relation_layer_bwd": (ctypes.c_int, [_PP, _PO, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t,
                                          _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "relation_decode_workspace_bytes": (ctypes.c_size_t, [_PP]),
    "relation_decode": (ctypes.c_int, [_PP, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "relation_decode_states": (ctypes.c_int, [_PP, _P, _P, _P, _P, ctypes.c_int32, ctypes.c_int32,
                                              ctypes.c_int32, _P, _P]),
    "relation_decode_merge": (ctypes.c_int, [_PP, ctypes.c_int32, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "relation_linear_fwd_workspace_bytes": (ctypes.c_size_t, [_PP]),
    "relation_linear_fwd": (ctypes.c_int, [_PP, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "relation_linear_bwd_workspace_bytes": (ctypes.c_size_t, [_PP]),
    "relation_linear_bwd": (ctypes.c_int, [_PP, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "relation_linear_gated_fwd_workspace_bytes": (ctypes.c_size_t, [_PP, ctypes.c_int32]),
    "relation_linear_gated_fwd": (ctypes.c_int, [_PP, _P, _P, _P, _P, _P, _P, ctypes.c_int32, ctypes.c_float, _P,
                                                 _P, _P, ctypes.c_size_t, _P]),
    "relation_linear_gated_bwd_workspace_bytes": (ctypes.c_size_t, [_PP, ctypes.c_int32]),
    "relation_linear_gated_bwd": (ctypes.c_int, [_PP, _P, _P, _P, _P, _P, _P, ctypes.c_int32, ctypes.c_float, _P,
                                                 _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "relation_profile_arm": (ctypes.c_int, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_void_p), ctypes.c_int]),
    "relation_profile_disarm": (ctypes.c_int, []),
    "relation_mfma_peak_flops": (ctypes.c_int64, [ctypes.c_int, ctypes.c_int]),
    "relation_mfma_peak_probe": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, _P, _P, _P]),
    "relation_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "relation_last_error": (ctypes.c_char_p, []),
    "relation_abi_version": (ctypes.c_int, []),
}

_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load librelation.so once. Raises if it has not been built: there is no
    fallback implementation."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"librelation.so not found at {path}; build it with "
                           "`python -m paper_2608_20172_amd.build`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int, what: str) -> None:
    if status != REL_OK:
        lib = load_library()
        msg = lib.relation_status_string(status).decode()
        detail = lib.relation_last_error().decode()
        raise RuntimeError(f"{what} failed: {msg} ({status}): {detail}")


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return REL_BF16
    if dt == torch.float32:
        return REL_F32
    raise TypeError(f"unsupported dtype {dt}; use torch.bfloat16 or torch.float32")


def make_problem(q: torch.Tensor, tau_s: float = TAU_S, scale: Optional[float] = None) -> RelProblem:
    if q.dim() != 4:
        raise ValueError("tensors must be [B, H, T, D]")
    B, H, T, D = q.shape
    sb, sh, st, sd = q.stride()
    if sd != 1:
        raise ValueError("the last dimension must be contiguous")
    return RelProblem(B, H, T, D, _dtype_code(q.dtype), 1, float(tau_s),
                      0.0 if scale is None else float(scale), sb, sh, st)


def _same_layout(ref: torch.Tensor, *ts: torch.Tensor) -> list:
    out = []
    for t in ts:
        if t.shape != ref.shape or t.dtype != ref.dtype or t.device != ref.device:
            raise ValueError("q, k, v (and o, dout) must share shape, dtype and device")
        if t.stride() != ref.stride():
            t = torch.empty_strided(ref.shape, ref.stride(), dtype=ref.dtype, device=ref.device).copy_(t)
        out.append(t)
    return out


def _lam_tensor(lam, device) -> torch.Tensor:
    if isinstance(lam, torch.Tensor):
        if lam.numel() != 1:
            raise ValueError("lambda must be a single scalar")
        return lam.detach().to(device=device, dtype=torch.float32).reshape(1).contiguous()
    return torch.tensor([float(lam)], dtype=torch.float32, device=device)


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _layout_like(q: torch.Tensor) -> torch.Tensor:
    # A dense [B, H, T, D] tensor keeps q's stride order; q's own strides are
    # reused so that every tensor shares (stride_b, stride_h, stride_t).
    return torch.empty_strided(q.shape, q.stride(), dtype=q.dtype, device=q.device)


def relation_fwd(q, k, v, lam, *, tau_s: float = TAU_S, scale: Optional[float] = None,
                 want_row_stat: bool = True, want_masses: bool = False, want_lse: bool = False):
    """Fused forward. Returns dict(o, row_stat, self_mass, exch_mass, exch_lse);
    outputs that were not requested are None."""
    lib = load_library()
    k, v = _same_layout(q, k, v)
    p = make_problem(q, tau_s, scale)
    B, H, T, D = q.shape
    dev = q.device
    lam_t = _lam_tensor(lam, dev)
    o = _layout_like(q)
    rows = lambda: torch.empty((B, H, T), dtype=torch.float32, device=dev)
    row_stat = rows() if want_row_stat else None
    self_mass = rows() if want_masses else None
    exch_mass = rows() if want_masses else None
    exch_lse = rows() if want_lse else None
    st = lib.relation_fwd(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(lam_t), _ptr(o),
                          _ptr(row_stat), _ptr(self_mass), _ptr(exch_mass), _ptr(exch_lse), _stream())
    _check(st, "relation_fwd")
    return {"o": o, "row_stat": row_stat, "self_mass": self_mass, "exch_mass": exch_mass,
            "exch_lse": exch_lse}


def relation_exchange_allocation(q, k, exch_lse, *, tau_s: float = TAU_S, scale: Optional[float] = None):
    """pi_ij = exp(E_ij - L^E_i) for j < i (dense [B, H, T, T] fp32)."""
    lib = load_library()
    (k,) = _same_layout(q, k)
    p = make_problem(q, tau_s, scale)
    B, H, T, D = q.shape
    pi = torch.empty((B, H, T, T), dtype=torch.float32, device=q.device)
    lse = exch_lse.contiguous().to(torch.float32)
    st = lib.relation_exchange_allocation(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(lse), _ptr(pi), _stream())
    _check(st, "relation_exchange_allocation")
    return pi


def relation_bwd_workspace_bytes(q, *, tau_s: float = TAU_S, scale: Optional[float] = None) -> int:
    lib = load_library()
    p = make_problem(q, tau_s, scale)
    return int(lib.relation_bwd_workspace_bytes(ctypes.byref(p)))


def relation_bwd(q, k, v, o, dout, lam, row_stat, *, tau_s: float = TAU_S,
                 scale: Optional[float] = None, want_dself: bool = False, workspace=None,
                 deterministic: bool = False):
    """Fused backward. Returns dict(dq, dk, dv, dlambda (1-element fp32 tensor), dself).
    deterministic=True calls relation_bwd_deterministic (bitwise repeatable dq)."""
    lib = load_library()
    k, v, o, dout = _same_layout(q, k, v, o, dout)
    p = make_problem(q, tau_s, scale)
    B, H, T, D = q.shape
    dev = q.device
    lam_t = _lam_tensor(lam, dev)
    dq, dk, dv = _layout_like(q), _layout_like(q), _layout_like(q)
    dlam = torch.empty((1,), dtype=torch.float32, device=dev)
    dself = torch.empty((B, H, T), dtype=torch.float32, device=dev) if want_dself else None
    nbytes = int(lib.relation_bwd_workspace_bytes(ctypes.byref(p)))
    if workspace is None or workspace.numel() * workspace.element_size() < nbytes:
        workspace = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=dev)
    rs = row_stat.contiguous()
    fn = lib.relation_bwd_deterministic if deterministic else lib.relation_bwd
    st = fn(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dout), _ptr(lam_t),
            _ptr(rs), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dlam), _ptr(dself),
            _ptr(workspace), workspace.numel() * workspace.element_size(), _stream())
    _check(st, "relation_bwd_deterministic" if deterministic else "relation_bwd")
    return {"dq": dq, "dk": dk, "dv": dv, "dlambda": dlam, "dself": dself}


def relation_bwd_noalloc(q, k, v, o, dout, lam, row_stat, *, tau_s: float = TAU_S,
                         scale: Optional[float] = None, want_dself: bool = False, out=None):
    """relation_bwd through the entry point that allocates nothing on the device
    (its scratch is the library's own per-device array). ``out`` may hold
    preallocated dq, dk, dv, dlambda (and dself) tensors. Returns the same dict."""
    lib = load_library()
    k, v, o, dout = _same_layout(q, k, v, o, dout)
    p = make_problem(q, tau_s, scale)
    B, H, T, D = q.shape
    dev = q.device
    lam_t = _lam_tensor(lam, dev)
    if out is None:
        out = {"dq": _layout_like(q), "dk": _layout_like(q), "dv": _layout_like(q),
               "dlambda": torch.empty((1,), dtype=torch.float32, device=dev),
               "dself": torch.empty((B, H, T), dtype=torch.float32, device=dev) if want_dself else None}
    rs = row_stat.contiguous()
    st = lib.relation_bwd_noalloc(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dout), _ptr(lam_t),
                                  _ptr(rs), _ptr(out["dq"]), _ptr(out["dk"]), _ptr(out["dv"]), _ptr(out["dlambda"]),
                                  _ptr(out.get("dself")), _stream())
    _check(st, "relation_bwd_noalloc")
    return out


def relation_fwd_materialized_workspace_bytes(q, *, tau_s: float = TAU_S,
                                              scale: Optional[float] = None) -> int:
    lib = load_library()
    p = make_problem(q, tau_s, scale)
    return int(lib.relation_fwd_materialized_workspace_bytes(ctypes.byref(p)))


def relation_fwd_materialized(q, k, v, lam, *, tau_s: float = TAU_S, scale: Optional[float] = None,
                              want_R: bool = False, want_F: bool = False, want_pi: bool = False,
                              want_masses: bool = False, workspace=None):
    """Materialised baseline. Returns dict(o, R, F, pi, self_mass, exch_mass)."""
    lib = load_library()
    k, v = _same_layout(q, k, v)
    p = make_problem(q, tau_s, scale)
    B, H, T, D = q.shape
    dev = q.device
    lam_t = _lam_tensor(lam, dev)
    o = _layout_like(q)
    mat = lambda: torch.empty((B, H, T, T), dtype=torch.float32, device=dev)
    rows = lambda: torch.empty((B, H, T), dtype=torch.float32, device=dev)
    R = mat() if want_R else None
    F = mat() if want_F else None
    pi = mat() if want_pi else None
    sm = rows() if want_masses else None
    em = rows() if want_masses else None
    nbytes = int(lib.relation_fwd_materialized_workspace_bytes(ctypes.byref(p)))
    if workspace is None or workspace.numel() * workspace.element_size() < nbytes:
        workspace = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=dev)
    st = lib.relation_fwd_materialized(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(lam_t), _ptr(o),
                                       _ptr(R), _ptr(F), _ptr(pi), _ptr(sm), _ptr(em), _ptr(workspace),
                                       workspace.numel() * workspace.element_size(), _stream())
    _check(st, "relation_fwd_materialized")
    return {"o": o, "R": R, "F": F, "pi": pi, "self_mass": sm, "exch_mass": em}


def relation_bwd_materialized_workspace_bytes(q, *, tau_s: float = TAU_S,
                                              scale: Optional[float] = None) -> int:
    lib = load_library()
    p = make_problem(q, tau_s, scale)
    return int(lib.relation_bwd_materialized_workspace_bytes(ctypes.byref(p)))


def relation_bwd_materialized(q, k, v, dout, lam, *, tau_s: float = TAU_S, scale: Optional[float] = None,
                              workspace=None):
    """Materialised backward baseline (every T x T tensor in HBM). Returns
    dict(dq, dk, dv, dlambda (1-element fp32 tensor))."""
    lib = load_library()
    k, v, dout = _same_layout(q, k, v, dout)
    p = make_problem(q, tau_s, scale)
    dev = q.device
    lam_t = _lam_tensor(lam, dev)
    dq, dk, dv = _layout_like(q), _layout_like(q), _layout_like(q)
    dlam = torch.empty((1,), dtype=torch.float32, device=dev)
    nbytes = int(lib.relation_bwd_materialized_workspace_bytes(ctypes.byref(p)))
    if workspace is None or workspace.numel() * workspace.element_size() < nbytes:
        workspace = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=dev)
    st = lib.relation_bwd_materialized(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(dout), _ptr(lam_t),
                                       _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dlam), _ptr(workspace),
                                       workspace.numel() * workspace.element_size(), _stream())
    _check(st, "relation_bwd_materialized")
    return {"dq": dq, "dk": dk, "dv": dv, "dlambda": dlam}


def make_layer_opts(pairing: Optional[str] = None, rope_base: float = ROPE_BASE,
                    transport: str = "full") -> RelLayerOpts:
    if pairing not in REL_GIVENS:
        raise ValueError("pairing must be None, 'A' or 'B'")
    if transport not in REL_TRANSPORT:
        raise ValueError("transport must be 'full' or 'exchange'")
    return RelLayerOpts(float(rope_base or 0.0), REL_GIVENS[pairing], REL_TRANSPORT[transport])


def _theta_tensor(theta, H: int, device):
    if theta is None:
        return None
    t = torch.as_tensor(theta, dtype=torch.float32, device=device).reshape(-1).contiguous()
    if t.numel() != H // 2:
        raise ValueError("theta must hold H/2 angles")
    return t


def _workspace(nbytes: int, ws, device):
    if nbytes == 0:
        return None
    if ws is None or ws.numel() * ws.element_size() < nbytes:
        ws = torch.empty((nbytes,), dtype=torch.uint8, device=device)
    return ws


def _layer_size(fn: str, q, pairing, rope_base, tau_s, scale) -> int:
    p, o = make_problem(q, tau_s, scale), make_layer_opts(pairing, rope_base)
    return int(getattr(load_library(), fn)(ctypes.byref(p), ctypes.byref(o)))


def relation_layer_saved_bytes(q, *, pairing: Optional[str] = None, rope_base: float = ROPE_BASE,
                               tau_s: float = TAU_S, scale: Optional[float] = None) -> int:
    return _layer_size("relation_layer_saved_bytes", q, pairing, rope_base, tau_s, scale)


def relation_layer_fwd_workspace_bytes(q, *, pairing: Optional[str] = None, rope_base: float = ROPE_BASE,
                                       tau_s: float = TAU_S, scale: Optional[float] = None) -> int:
    return _layer_size("relation_layer_fwd_workspace_bytes", q, pairing, rope_base, tau_s, scale)


def relation_layer_bwd_workspace_bytes(q, *, pairing: Optional[str] = None, rope_base: float = ROPE_BASE,
                                       tau_s: float = TAU_S, scale: Optional[float] = None) -> int:
    return _layer_size("relation_layer_bwd_workspace_bytes", q, pairing, rope_base, tau_s, scale)


def _nbytes(t) -> int:
    return 0 if t is None else t.numel() * t.element_size()


def relation_layer_fwd(q, k, v, lam, theta=None, *, pairing: Optional[str] = None,
                       rope_base: float = ROPE_BASE, transport: str = "full", tau_s: float = TAU_S,
                       scale: Optional[float] = None, keep_saved: bool = True, workspace=None):
    """Layer forward: RoPE on q, k (rope_base 0: off), Givens mixing of v over
    head pairs ("A", "B" or None) with angles ``theta`` [H/2], then the fused
    operator. Any head width up to 128. Returns dict(o, row_stat, saved):
    ``saved`` (a uint8 device tensor, or None) holds the prepared operands for
    relation_layer_bwd; with keep_saved=False it is None and the backward pass
    prepares them again."""
    lib = load_library()
    k, v = _same_layout(q, k, v)
    p = make_problem(q, tau_s, scale)
    opts = make_layer_opts(pairing, rope_base, transport)
    dev = q.device
    lam_t = _lam_tensor(lam, dev)
    th = _theta_tensor(theta, q.shape[1], dev) if pairing else None
    o = _layout_like(q)
    rs = torch.empty(q.shape[:3], dtype=torch.float32, device=dev)
    nsaved = int(lib.relation_layer_saved_bytes(ctypes.byref(p), ctypes.byref(opts)))
    saved = torch.empty((nsaved,), dtype=torch.uint8, device=dev) if keep_saved and nsaved else None
    ws = None if saved is not None else _workspace(
        int(lib.relation_layer_fwd_workspace_bytes(ctypes.byref(p), ctypes.byref(opts))), workspace, dev)
    st = lib.relation_layer_fwd(ctypes.byref(p), ctypes.byref(opts), _ptr(q), _ptr(k), _ptr(v), _ptr(lam_t),
                                _ptr(th), _ptr(o), _ptr(rs), _ptr(saved), _nbytes(saved), _ptr(ws), _nbytes(ws),
                                _stream())
    _check(st, "relation_layer_fwd")
    return {"o": o, "row_stat": rs, "saved": saved}


def relation_layer_bwd(q, k, v, o, dout, lam, row_stat, theta=None, *, saved=None, pairing: Optional[str] = None,
                       rope_base: float = ROPE_BASE, transport: str = "full", tau_s: float = TAU_S,
                       scale: Optional[float] = None, workspace=None):
    """Layer backward; ``saved`` is the forward call's (None: recompute).
    Returns dict(dq, dk, dv, dlambda [1], dtheta [H/2] or None)."""
    lib = load_library()
    k, v, o, dout = _same_layout(q, k, v, o, dout)
    p = make_problem(q, tau_s, scale)
    opts = make_layer_opts(pairing, rope_base, transport)
    dev = q.device
    lam_t = _lam_tensor(lam, dev)
    H = q.shape[1]
    th = _theta_tensor(theta, H, dev) if pairing else None
    rs = row_stat.contiguous()
    dq, dk, dv = _layout_like(q), _layout_like(q), _layout_like(q)
    dlam = torch.empty((1,), dtype=torch.float32, device=dev)
    dth = torch.empty((H // 2,), dtype=torch.float32, device=dev) if pairing else None
    nbytes = int(lib.relation_layer_bwd_workspace_bytes(ctypes.byref(p), ctypes.byref(opts)))
    ws = _workspace(max(nbytes, 1), workspace, dev)
    st = lib.relation_layer_bwd(ctypes.byref(p), ctypes.byref(opts), _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                                _ptr(dout), _ptr(lam_t), _ptr(th), _ptr(rs), _ptr(saved), _nbytes(saved),
                                _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dlam), _ptr(dth), _ptr(ws), _nbytes(ws),
                                _stream())
    _check(st, "relation_layer_bwd")
    return {"dq": dq, "dk": dk, "dv": dv, "dlambda": dlam, "dtheta": dth}


def _decode_io(q, k_cache, v_cache, lengths, tau_s, scale):
    v_cache = _same_layout(k_cache, v_cache)[0]
    B, H, T, D = k_cache.shape
    if q.shape != (B, H, D) or q.dtype != k_cache.dtype:
        raise ValueError("q must be [B, H, D] with the caches' dtype")
    q = q.contiguous()
    lengths = torch.as_tensor(lengths, dtype=torch.int32, device=q.device).reshape(B).contiguous()
    return q, k_cache, v_cache, lengths, make_problem(k_cache, tau_s, scale)


def relation_decode(q, k_cache, v_cache, lengths, lam, *, tau_s: float = TAU_S, scale: Optional[float] = None,
                    workspace=None):
    """One decode step: q [B, H, D] of the new tokens, caches [B, H, Tmax, D]
    holding lengths[b] entries each (the new token's own entry last).
    Returns dict(o [B, H, D], row_stat [B, H])."""
    lib = load_library()
    q, k_cache, v_cache, lengths, p = _decode_io(q, k_cache, v_cache, lengths, tau_s, scale)
    dev = q.device
    lam_t = _lam_tensor(lam, dev)
    o = torch.empty_like(q)
    rs = torch.empty(q.shape[:2], dtype=torch.float32, device=dev)
    ws = _workspace(max(1, int(lib.relation_decode_workspace_bytes(ctypes.byref(p)))), workspace, dev)
    st = lib.relation_decode(ctypes.byref(p), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(lengths), _ptr(lam_t),
                             _ptr(o), _ptr(rs), _ptr(ws), _nbytes(ws), _stream())
    _check(st, "relation_decode")
    return {"o": o, "row_stat": rs}


def relation_decode_states(q, k_cache, v_cache, lengths, key_begin: int, key_end: int, nstates: int = 1, *,
                           tau_s: float = TAU_S, scale: Optional[float] = None):
    """Exchange scan states [nstates, B*H, D + 2] (m, l, z) of cache keys
    [key_begin, key_end) for the new tokens' rows."""
    lib = load_library()
    q, k_cache, v_cache, lengths, p = _decode_io(q, k_cache, v_cache, lengths, tau_s, scale)
    B, H, _, D = k_cache.shape
    states = torch.empty((nstates, B * H, D + 2), dtype=torch.float32, device=q.device)
    st = lib.relation_decode_states(ctypes.byref(p), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(lengths),
                                    int(key_begin), int(key_end), int(nstates), _ptr(states), _stream())
    _check(st, "relation_decode_states")
    return states


def relation_decode_merge(states, q, k_cache, v_cache, lengths, lam, *, tau_s: float = TAU_S,
                          scale: Optional[float] = None):
    """Merge states [n, B*H, D + 2] with the Self entry; dict(o, row_stat)."""
    lib = load_library()
    q, k_cache, v_cache, lengths, p = _decode_io(q, k_cache, v_cache, lengths, tau_s, scale)
    dev = q.device
    states = states.to(dtype=torch.float32).contiguous()
    lam_t = _lam_tensor(lam, dev)
    o = torch.empty_like(q)
    rs = torch.empty(q.shape[:2], dtype=torch.float32, device=dev)
    st = lib.relation_decode_merge(ctypes.byref(p), int(states.shape[0]), _ptr(states), _ptr(q), _ptr(k_cache),
                                   _ptr(v_cache), _ptr(lengths), _ptr(lam_t), _ptr(o), _ptr(rs), _stream())
    _check(st, "relation_decode_merge")
    return {"o": o, "row_stat": rs}


def relation_linear_fwd(p1, p2, v, g, *, tau_s: float = TAU_S, scale: Optional[float] = None,
                        want_state: bool = False, workspace=None):
    """Linear Relation forward over [B, H, T, D] tensors; g is the fp32
    log-retention. Returns dict(o, state (the [B, H, D, D] state after the last
    token, or None))."""
    lib = load_library()
    p2, v = _same_layout(p1, p2, v)
    p = make_problem(p1, tau_s, scale)
    dev = p1.device
    g = g.to(device=dev, dtype=torch.float32).contiguous()
    if g.shape != p1.shape:
        raise ValueError("g must have the shape of p1")
    o = _layout_like(p1)
    B, H, T, D = p1.shape
    state = torch.empty((B, H, D, D), dtype=torch.float32, device=dev) if want_state else None
    ws = _workspace(max(1, int(lib.relation_linear_fwd_workspace_bytes(ctypes.byref(p)))), workspace, dev)
    st = lib.relation_linear_fwd(ctypes.byref(p), _ptr(p1), _ptr(p2), _ptr(v), _ptr(g), _ptr(o), _ptr(state),
                                 _ptr(ws), _nbytes(ws), _stream())
    _check(st, "relation_linear_fwd")
    return {"o": o, "state": state}


def relation_linear_bwd(p1, p2, v, g, dout, *, tau_s: float = TAU_S, scale: Optional[float] = None,
                        workspace=None):
    """Linear Relation backward. Returns dict(dp1, dp2, dv, dg (fp32))."""
    lib = load_library()
    p2, v, dout = _same_layout(p1, p2, v, dout)
    p = make_problem(p1, tau_s, scale)
    dev = p1.device
    g = g.to(device=dev, dtype=torch.float32).contiguous()
    dp1, dp2, dv = _layout_like(p1), _layout_like(p1), _layout_like(p1)
    dg = torch.empty(p1.shape, dtype=torch.float32, device=dev)
    ws = _workspace(max(1, int(lib.relation_linear_bwd_workspace_bytes(ctypes.byref(p)))), workspace, dev)
    st = lib.relation_linear_bwd(ctypes.byref(p), _ptr(p1), _ptr(p2), _ptr(v), _ptr(g), _ptr(dout), _ptr(dp1),
                                 _ptr(dp2), _ptr(dv), _ptr(dg), _ptr(ws), _nbytes(ws), _stream())
    _check(st, "relation_linear_bwd")
    return {"dp1": dp1, "dp2": dp2, "dv": dv, "dg": dg}


def _gate_params(a_log, dt_bias, p1):
    H, D = p1.shape[1], p1.shape[3]
    out = []
    for name, x in (("a_log", a_log), ("dt_bias", dt_bias)):
        x = x.to(device=p1.device, dtype=torch.float32).contiguous()
        if tuple(x.shape) != (H, D):
            raise ValueError(f"{name} must have shape [H, D] = [{H}, {D}]")
        out.append(x)
    return out


def relation_linear_gated_fwd(p1, p2, v, r, a_log, dt_bias, *, rope_dim: int = 0, rope_base: float = 1.0e4,
                              tau_s: float = TAU_S, scale: Optional[float] = None, want_state: bool = False,
                              workspace=None):
    """Linear Relation forward with the retention gate of eq. 15 formed in the
    kernels from r ([B, H, T, D] fp32) and a_log, dt_bias ([H, D] fp32), and
    RoPE over the first rope_dim channels of p1, p2 (0: none).
    Returns dict(o, state)."""
    lib = load_library()
    p2, v = _same_layout(p1, p2, v)
    p = make_problem(p1, tau_s, scale)
    dev = p1.device
    r = r.to(device=dev, dtype=torch.float32).contiguous()
    if r.shape != p1.shape:
        raise ValueError("r must have the shape of p1")
    a_log, dt_bias = _gate_params(a_log, dt_bias, p1)
    o = _layout_like(p1)
    B, H, T, D = p1.shape
    state = torch.empty((B, H, D, D), dtype=torch.float32, device=dev) if want_state else None
    ws = _workspace(max(1, int(lib.relation_linear_gated_fwd_workspace_bytes(ctypes.byref(p), rope_dim))),
                    workspace, dev)
    st = lib.relation_linear_gated_fwd(ctypes.byref(p), _ptr(p1), _ptr(p2), _ptr(v), _ptr(r), _ptr(a_log),
                                       _ptr(dt_bias), rope_dim, rope_base, _ptr(o), _ptr(state), _ptr(ws),
                                       _nbytes(ws), _stream())
    _check(st, "relation_linear_gated_fwd")
    return {"o": o, "state": state}


def relation_linear_gated_bwd(p1, p2, v, r, a_log, dt_bias, dout, *, rope_dim: int = 0, rope_base: float = 1.0e4,
                              tau_s: float = TAU_S, scale: Optional[float] = None, workspace=None):
    """Backward of relation_linear_gated_fwd. Returns dict(dp1, dp2, dv, dr
    (fp32), da_log, ddt_bias ([H, D] fp32))."""
    lib = load_library()
    p2, v, dout = _same_layout(p1, p2, v, dout)
    p = make_problem(p1, tau_s, scale)
    dev = p1.device
    r = r.to(device=dev, dtype=torch.float32).contiguous()
    a_log, dt_bias = _gate_params(a_log, dt_bias, p1)
    dp1, dp2, dv = _layout_like(p1), _layout_like(p1), _layout_like(p1)
    dr = torch.empty(p1.shape, dtype=torch.float32, device=dev)
    da_log, ddt_bias = torch.empty_like(a_log), torch.empty_like(dt_bias)
    ws = _workspace(max(1, int(lib.relation_linear_gated_bwd_workspace_bytes(ctypes.byref(p), rope_dim))),
                    workspace, dev)
    st = lib.relation_linear_gated_bwd(ctypes.byref(p), _ptr(p1), _ptr(p2), _ptr(v), _ptr(r), _ptr(a_log),
                                       _ptr(dt_bias), rope_dim, rope_base, _ptr(dout), _ptr(dp1), _ptr(dp2),
                                       _ptr(dv), _ptr(dr), _ptr(da_log), _ptr(ddt_bias), _ptr(ws), _nbytes(ws),
                                       _stream())
    _check(st, "relation_linear_gated_bwd")
    return {"dp1": dp1, "dp2": dp2, "dv": dv, "dr": dr, "da_log": da_log, "ddt_bias": ddt_bias}


def relation_profile_arm(kernel: str, events: list) -> None:
    """Record each listed torch.cuda.Event pair around successive launches of
    ``kernel`` ("fwd" or "bwd"); events = [start0, stop0, start1, stop1, ...]."""
    lib = load_library()
    arr = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
    _check(lib.relation_profile_arm(kernel.encode(), arr, len(events) // 2), "relation_profile_arm")
    relation_profile_arm._keep = arr


def relation_profile_disarm() -> int:
    return int(load_library().relation_profile_disarm())


class _RelationFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, lam, tau_s, scale):
        out = relation_fwd(q, k, v, lam, tau_s=tau_s, scale=scale)
        ctx.save_for_backward(q, k, v, out["o"], lam, out["row_stat"])
        ctx.tau_s, ctx.scale = tau_s, scale
        return out["o"]

    @staticmethod
    def backward(ctx, dout):
        q, k, v, o, lam, row_stat = ctx.saved_tensors
        g = relation_bwd(q, k, v, o, dout.contiguous() if dout.stride() != q.stride() else dout, lam,
                         row_stat, tau_s=ctx.tau_s, scale=ctx.scale)
        dlam = g["dlambda"].reshape(lam.shape).to(lam.dtype)
        return g["dq"], g["dk"], g["dv"], dlam, None, None


def relation(q, k, v, lam, tau_s: float = TAU_S, scale: Optional[float] = None) -> torch.Tensor:
    """Differentiable causal Full Relation over [B, H, T, D] tensors (fused
    FlashRelation kernels). ``lam`` is a scalar tensor (the layer's lambda)."""
    if not isinstance(lam, torch.Tensor):
        lam = torch.tensor(float(lam), dtype=torch.float32, device=q.device)
    return _RelationFn.apply(q, k, v, lam, tau_s, scale)

