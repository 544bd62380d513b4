"""C-ABI checks that need no GPU: the library loads, exports every entry point
declared in include/relation.h, and validates arguments on the host before
any HIP call. With valid arguments and no device, a call reaches the launch
and reports REL_ERR_HIP."""
import ctypes
import os
import re

import pytest

from paper_2608_20172_amd import binding as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "relation.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(R.LIB_PATH):
        from paper_2608_20172_amd import build
        build.build()
    return R.load_library()


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(relation_\w+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    syms = declared_symbols()
    assert len(syms) >= 9
    for s in syms:
        assert hasattr(lib, s), f"{s} not exported"
    assert lib.relation_abi_version() == 1


def prob(B=1, H=2, T=128, D=64, dtype=R.REL_BF16, causal=1, tau=2.0, scale=0.0, sb=None, sh=None, st=None):
    st = D if st is None else st
    sh = T * st if sh is None else sh
    sb = H * sh if sb is None else sb
    return R.RelProblem(B, H, T, D, dtype, causal, tau, scale, sb, sh, st)


BASE = 0x7F0000000000
MB = 1 << 24


def ptrs(n):
    return [BASE + i * MB for i in range(n)]


def fwd(lib, p, q=None, k=None, v=None, lam=None, o=None, rs=None, sm=None, em=None, lse=None):
    a = ptrs(5)
    q = a[0] if q is None else q
    k = a[1] if k is None else k
    v = a[2] if v is None else v
    lam = a[3] if lam is None else lam
    o = a[4] if o is None else o
    return lib.relation_fwd(ctypes.byref(p) if p is not None else None, q, k, v, lam, o, rs, sm, em, lse, None)


def test_valid_call_reaches_launch(lib):
    assert fwd(lib, prob()) == R.REL_ERR_HIP
    assert fwd(lib, prob(D=96)) == R.REL_ERR_HIP  # bf16 width 96
    assert b"device" in lib.relation_last_error() or b"HIP" in lib.relation_last_error()


@pytest.mark.parametrize("mut,code", [
    (dict(D=48), R.REL_ERR_UNSUPPORTED),
    (dict(D=96, dtype=R.REL_F32), R.REL_ERR_UNSUPPORTED),   # 96 is tiled for bf16 only
    (dict(D=256), R.REL_ERR_UNSUPPORTED),
    (dict(causal=0), R.REL_ERR_UNSUPPORTED),
    (dict(dtype=7), R.REL_ERR_UNSUPPORTED),
    (dict(tau=0.0), R.REL_ERR_INVALID_ARG),
    (dict(tau=-1.0), R.REL_ERR_INVALID_ARG),
    (dict(tau=float("inf")), R.REL_ERR_INVALID_ARG),
    (dict(scale=float("nan")), R.REL_ERR_INVALID_ARG),
    (dict(T=-1), R.REL_ERR_INVALID_ARG),
    (dict(st=60), R.REL_ERR_INVALID_ARG),          # stride_t < D
    (dict(st=68), R.REL_ERR_INVALID_ARG),          # not a multiple of 16 bytes
    (dict(sh=64), R.REL_ERR_INVALID_ARG),          # heads overlap rows
    (dict(T=(1 << 24) + 8), R.REL_ERR_UNSUPPORTED),
    (dict(T=1 << 22, st=256), R.REL_ERR_UNSUPPORTED),  # one head spans 2 GiB of bf16
])
def test_problem_validation(lib, mut, code):
    assert fwd(lib, prob(**mut)) == code


def test_null_and_alignment(lib):
    assert fwd(lib, None) == R.REL_ERR_INVALID_ARG
    p = prob()
    a = ptrs(5)
    assert lib.relation_fwd(ctypes.byref(p), 0, a[1], a[2], a[3], a[4], None, None, None, None, None) == R.REL_ERR_INVALID_ARG
    assert fwd(lib, p, q=BASE + 8) == R.REL_ERR_INVALID_ARG       # q not 16-byte aligned
    assert fwd(lib, p, lam=0) == R.REL_ERR_INVALID_ARG             # lambda required
    assert fwd(lib, p, rs=BASE + 5 * MB + 2) == R.REL_ERR_INVALID_ARG  # row_stat misaligned


def test_empty_problem_is_ok(lib):
    for mut in (dict(B=0), dict(H=0), dict(T=0)):
        assert fwd(lib, prob(**mut), q=0, k=0, v=0, o=0) == R.REL_OK


def test_output_aliasing(lib):
    p = prob()
    a = ptrs(5)
    assert fwd(lib, p, o=a[0]) == R.REL_ERR_INVALID_ARG                  # o == q
    assert fwd(lib, p, o=a[0] + 128) == R.REL_ERR_INVALID_ARG            # o shifted one row into q
    assert fwd(lib, p, rs=a[1]) == R.REL_ERR_INVALID_ARG                 # row stat inside k
    assert fwd(lib, p, rs=BASE + 5 * MB, sm=BASE + 5 * MB) == R.REL_ERR_INVALID_ARG
    # interleaved, element-disjoint layouts are accepted: q and o as the two
    # halves of every row of a [B, H, T, 2, D] buffer (stride_t = 2 D)
    p2 = prob(st=128, sh=128 * 128)
    assert fwd(lib, p2, q=a[0], o=a[0] + 64 * 2) == R.REL_ERR_HIP
    # but shifting o by one element makes the halves overlap
    assert fwd(lib, p2, q=a[0], o=a[0] + 62 * 2 + 16) == R.REL_ERR_INVALID_ARG


def test_bwd_workspace_and_dtype_limits(lib):
    p = prob(T=300)
    need = lib.relation_bwd_workspace_bytes(ctypes.byref(p))
    assert 0 < need < 1 << 20  # per-workgroup dlambda partials only
    a = ptrs(16)
    args = [ctypes.byref(p), a[0], a[1], a[2], a[3], a[4], a[5], a[6], a[7], a[8], a[9], a[10], None]
    assert lib.relation_bwd(*args, a[11], need - 1, None) == R.REL_ERR_WORKSPACE
    assert lib.relation_bwd(*args, None, need, None) == R.REL_ERR_WORKSPACE
    assert lib.relation_bwd(*args, a[11], need, None) == R.REL_ERR_HIP
    p32 = prob(T=300, D=128, dtype=R.REL_F32, st=128)
    n32 = lib.relation_bwd_workspace_bytes(ctypes.byref(p32))
    args32 = [ctypes.byref(p32)] + args[1:]
    assert lib.relation_bwd(*args32, a[11], n32, None) == R.REL_ERR_HIP  # supported, reaches launch
    assert lib.relation_bwd_workspace_bytes(None) == 0


def test_materialized_workspace(lib):
    p = prob(T=256)
    need = lib.relation_fwd_materialized_workspace_bytes(ctypes.byref(p))
    assert need >= 2 * 256 * 256 * (4 + 2)
    a = ptrs(12)
    assert lib.relation_fwd_materialized(ctypes.byref(p), a[0], a[1], a[2], a[3], a[4], None, None, None,
                                         None, None, a[5], need - 1, None) == R.REL_ERR_WORKSPACE
    assert lib.relation_fwd_materialized(ctypes.byref(p), a[0], a[1], a[2], a[3], a[4], None, None, None,
                                         None, None, a[5], need, None) == R.REL_ERR_HIP


def test_materialized_backward_workspace(lib):
    p = prob(T=256)
    need = lib.relation_bwd_materialized_workspace_bytes(ctypes.byref(p))
    # U and H in fp32, dU and F in bf16, one fp32 dlambda term per row
    assert need >= 2 * 256 * 256 * (2 * 4 + 2 * 2) + 2 * 256 * 4 + 256 * 4
    a = ptrs(12)
    call = lambda pp, ws, n: lib.relation_bwd_materialized(ctypes.byref(pp), a[0], a[1], a[2], a[3], a[4],
                                                           a[5], a[6], a[7], a[8], ws, n, None)
    assert call(p, a[9], need - 1) == R.REL_ERR_WORKSPACE
    assert call(p, None, need) == R.REL_ERR_WORKSPACE
    assert call(p, a[9], need) == R.REL_ERR_HIP  # valid request; fails only at the device
    # T x T per head must stay within 2^31 elements
    big = prob(B=1, H=1, T=46341)
    assert call(big, a[9], 1 << 45) == R.REL_ERR_UNSUPPORTED
    assert lib.relation_bwd_materialized_workspace_bytes(ctypes.byref(prob(T=0))) == 0
    assert lib.relation_bwd_materialized_workspace_bytes(None) == 0


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4):
        assert lib.relation_status_string(code)
    assert lib.relation_status_string(-99) == b"unknown status"


def test_injected_launch_failure_raises(lib, monkeypatch):
    monkeypatch.setenv("RELATION_TEST_FAIL_LAUNCH", "1")
    assert fwd(lib, prob()) == R.REL_ERR_HIP
    assert b"injected" in lib.relation_last_error()
    with pytest.raises(RuntimeError, match="relation_fwd failed"):
        R._check(R.REL_ERR_HIP, "relation_fwd")


# ---------------------------------------------------------------------------
# layer entry points (RoPE, Givens mixing, padded head widths)
# ---------------------------------------------------------------------------
def lopts(rope=1.0e4, givens=1, transport=0):
    return R.RelLayerOpts(rope, givens, transport)


def layer_fwd(lib, p, o, theta=True, ws_bytes=None, saved=None, saved_bytes=0):
    a = ptrs(8)
    need = lib.relation_layer_fwd_workspace_bytes(ctypes.byref(p), ctypes.byref(o))
    n = need if ws_bytes is None else ws_bytes
    return lib.relation_layer_fwd(ctypes.byref(p), ctypes.byref(o), a[0], a[1], a[2], a[3],
                                  a[4] if theta else None, a[5], a[6], saved, saved_bytes, a[7], n, None)


def test_layer_workspace_sizes(lib):
    p = prob(B=2, H=4, T=100, D=60, st=60)
    es, DP = 2, 64
    tensor = 2 * 4 * 100 * DP * es
    sv = lib.relation_layer_saved_bytes(ctypes.byref(p), ctypes.byref(lopts()))
    fw = lib.relation_layer_fwd_workspace_bytes(ctypes.byref(p), ctypes.byref(lopts()))
    bw = lib.relation_layer_bwd_workspace_bytes(ctypes.byref(p), ctypes.byref(lopts()))
    # saved: rotated q, k, mixed v and the padded output; the [T, D/2] cos/sin table
    assert sv >= 4 * tensor + 100 * 30 * 8 and fw == sv
    # backward adds padded dout, three padded gradients, one dtheta term per (pair, b, t)
    assert bw >= sv + 4 * tensor + 2 * 2 * 100 * 4
    # a pass-through layer (no RoPE, no mixing, tiled width, contiguous) prepares nothing
    p64 = prob(B=2, H=4, T=100, D=64)
    assert lib.relation_layer_saved_bytes(ctypes.byref(p64), ctypes.byref(lopts(0.0, 0))) == 0
    assert lib.relation_layer_saved_bytes(ctypes.byref(p64), ctypes.byref(lopts(1.0e4, 0))) > 0
    assert lib.relation_layer_fwd_workspace_bytes(ctypes.byref(prob(T=0)), ctypes.byref(lopts())) == 0
    assert lib.relation_layer_fwd_workspace_bytes(None, ctypes.byref(lopts())) == 0
    assert lib.relation_layer_fwd_workspace_bytes(ctypes.byref(p), None) == 0


@pytest.mark.parametrize("pmut,omut,code", [
    (dict(D=60, st=60), {}, R.REL_ERR_HIP),             # paper width 60, rows 120 bytes apart: accepted
    (dict(D=48, st=48), {}, R.REL_ERR_HIP),
    (dict(D=80, st=80), {}, R.REL_ERR_HIP),
    (dict(D=130, st=130), {}, R.REL_ERR_UNSUPPORTED),
    (dict(D=61, st=61), {}, R.REL_ERR_INVALID_ARG),    # RoPE needs an even width
    (dict(D=61, st=61), dict(rope=0.0), R.REL_ERR_HIP),
    (dict(H=3), {}, R.REL_ERR_INVALID_ARG),            # Givens needs paired heads
    (dict(H=3), dict(givens=0), R.REL_ERR_HIP),
    ({}, dict(givens=3), R.REL_ERR_INVALID_ARG),
    ({}, dict(transport=2), R.REL_ERR_INVALID_ARG),
    ({}, dict(transport=1), R.REL_ERR_HIP),           # exchange-only ablation
    ({}, dict(rope=0.5), R.REL_ERR_INVALID_ARG),
    ({}, dict(rope=float("nan")), R.REL_ERR_INVALID_ARG),
    (dict(causal=0), {}, R.REL_ERR_UNSUPPORTED),
])
def test_layer_validation(lib, pmut, omut, code):
    assert layer_fwd(lib, prob(**pmut), lopts(**omut)) == code


def test_layer_arguments(lib):
    p = prob(D=60, st=60)
    o = lopts()
    assert layer_fwd(lib, p, o, theta=False) == R.REL_ERR_INVALID_ARG      # angles required
    assert layer_fwd(lib, p, lopts(givens=0), theta=False) == R.REL_ERR_HIP
    assert layer_fwd(lib, p, o, ws_bytes=16) == R.REL_ERR_WORKSPACE
    sv = lib.relation_layer_saved_bytes(ctypes.byref(p), ctypes.byref(o))
    saved = BASE + 12 * MB
    assert layer_fwd(lib, p, o, ws_bytes=0, saved=saved, saved_bytes=sv - 1) == R.REL_ERR_WORKSPACE
    assert layer_fwd(lib, p, o, ws_bytes=0, saved=saved, saved_bytes=sv) == R.REL_ERR_HIP  # no workspace needed
    assert layer_fwd(lib, p, o, saved=saved + 8, saved_bytes=sv) == R.REL_ERR_INVALID_ARG  # misaligned
    a = ptrs(8)
    assert lib.relation_layer_fwd(ctypes.byref(p), ctypes.byref(o), a[0], a[1], a[2], a[3], a[4], a[0],
                                  a[6], None, 0, a[7], 1 << 30, None) == R.REL_ERR_INVALID_ARG  # out == q
    # backward: a valid request reaches the device; a short workspace does not
    need = lib.relation_layer_bwd_workspace_bytes(ctypes.byref(p), ctypes.byref(o))
    b = ptrs(16)

    def bwd(saved_ptr, saved_n, ws_n, dtheta=True):
        args = b[:8] + [saved_ptr, saved_n] + b[8:11] + [b[11], b[12] if dtheta else None, b[13], ws_n]
        return lib.relation_layer_bwd(ctypes.byref(p), ctypes.byref(o), *args, None)

    assert bwd(None, 0, need - 1) == R.REL_ERR_WORKSPACE
    assert bwd(None, 0, need) == R.REL_ERR_HIP
    assert bwd(None, 0, need, dtheta=False) == R.REL_ERR_INVALID_ARG     # dtheta required
    # with the forward's saved buffer the backward needs less workspace
    assert bwd(b[14], sv, need - sv) == R.REL_ERR_HIP
    assert bwd(b[14], sv, need - sv - 1) == R.REL_ERR_WORKSPACE
    assert bwd(b[14], sv - 1, need) == R.REL_ERR_WORKSPACE
    # empty problem with no scalar outputs: nothing to launch
    pe = prob(B=0)
    assert lib.relation_layer_bwd(ctypes.byref(pe), ctypes.byref(o), *([None] * 8), None, 0, *([None] * 5), None,
                                  0, None) == R.REL_OK


# ---------------------------------------------------------------------------
# decode step
# ---------------------------------------------------------------------------
def test_decode_validation(lib):
    p = prob(B=2, H=3, T=1000, D=64)
    need = lib.relation_decode_workspace_bytes(ctypes.byref(p))
    # one state (2 + D floats) per 256-key slice of the history and (b, h) row
    assert need >= 4 * 2 * 3 * 66 * 4
    a = ptrs(10)
    call = lambda pp, ws_n, **kw: lib.relation_decode(ctypes.byref(pp), kw.get("q", a[0]), a[1], a[2], a[3], a[4],
                                                       kw.get("out", a[5]), None, a[6], ws_n, None)
    assert call(p, need) == R.REL_ERR_HIP                 # valid: reaches the device
    assert call(p, need - 1) == R.REL_ERR_WORKSPACE
    assert call(p, need, q=a[0] + 8) == R.REL_ERR_INVALID_ARG   # q not 16-byte aligned
    assert call(p, need, out=a[0]) == R.REL_ERR_INVALID_ARG     # out overlaps q
    assert call(prob(B=2, H=3, T=0, D=64), 1 << 20) == R.REL_ERR_INVALID_ARG  # no room for the new entry
    assert call(prob(B=0, H=3, T=8, D=64), 0) == R.REL_OK
    assert call(prob(D=48), 1 << 20) == R.REL_ERR_UNSUPPORTED
    # states: the key range must lie in the cache, nstates >= 1
    st = lambda k0, k1, n: lib.relation_decode_states(ctypes.byref(p), a[0], a[1], a[2], a[3], k0, k1, n, a[7], None)
    assert st(0, 1000, 4) == R.REL_ERR_HIP
    assert st(-1, 10, 1) == R.REL_ERR_INVALID_ARG
    assert st(10, 1001, 1) == R.REL_ERR_INVALID_ARG
    assert st(20, 10, 1) == R.REL_ERR_INVALID_ARG
    assert st(0, 10, 0) == R.REL_ERR_INVALID_ARG
    mg = lambda n, states: lib.relation_decode_merge(ctypes.byref(p), n, states, a[0], a[1], a[2], a[3], a[4],
                                                     a[5], None, None)
    assert mg(3, a[7]) == R.REL_ERR_HIP
    assert mg(0, None) == R.REL_ERR_HIP                   # no states: a pure Self row
    assert mg(-1, a[7]) == R.REL_ERR_INVALID_ARG
    assert mg(2, a[5]) == R.REL_ERR_INVALID_ARG           # states inside out


def test_noalloc_backward_validates_before_any_hip_call(lib):
    """The no-allocation backward rejects a problem whose scratch exceeds its
    per-device array with REL_ERR_WORKSPACE, before touching the device; a
    valid problem reaches the device (no GPU here: REL_ERR_HIP)."""
    a = ptrs(12)
    cap = lib.relation_bwd_noalloc_max_scratch_bytes()
    assert cap == 32 << 20
    big = prob(B=1, H=64, T=1 << 16, D=32)
    assert lib.relation_bwd_workspace_bytes(ctypes.byref(big)) > cap
    st = lib.relation_bwd_noalloc(ctypes.byref(big), *a[:11], None, None)
    assert st == R.REL_ERR_WORKSPACE
    assert b"scratch" in lib.relation_last_error()
    small = prob()
    assert lib.relation_bwd_workspace_bytes(ctypes.byref(small)) <= cap
    assert lib.relation_bwd_noalloc(ctypes.byref(small), *a[:11], None, None) == R.REL_ERR_HIP
    # an invalid problem is reported as such, whatever its size
    assert lib.relation_bwd_noalloc(ctypes.byref(prob(D=48)), *a[:11], None, None) == R.REL_ERR_UNSUPPORTED


def test_linear_widths_and_workspace(lib):
    """Linear Relation takes widths 32, 64 and 128 forward and backward (128
    as four 64-channel problems, whose backward workspace holds at least qt,
    kt and eight partial-gradient planes of fp32 per token); other widths are
    refused before any device work, and valid calls reach the launch."""
    a = ptrs(10)
    for D in (32, 64, 128):
        p = prob(B=2, H=3, T=300, D=D)
        fws = lib.relation_linear_fwd_workspace_bytes(ctypes.byref(p))
        bws = lib.relation_linear_bwd_workspace_bytes(ctypes.byref(p))
        assert fws > 0 and bws > fws
        if D == 128:
            assert bws >= 10 * 2 * 3 * 300 * 128 * 4
        st = lib.relation_linear_bwd(ctypes.byref(p), a[0], a[1], a[2], a[3], a[4], a[5], a[6], a[7], a[8],
                                     a[9], bws, None)
        assert st == R.REL_ERR_HIP
        st = lib.relation_linear_bwd(ctypes.byref(p), a[0], a[1], a[2], a[3], a[4], a[5], a[6], a[7], a[8],
                                     a[9], bws - 1, None)
        assert st == R.REL_ERR_WORKSPACE
    for D in (48, 80, 96):
        p = prob(B=1, H=1, T=64, D=D)
        assert lib.relation_linear_bwd_workspace_bytes(ctypes.byref(p)) == 0
        st = lib.relation_linear_bwd(ctypes.byref(p), a[0], a[1], a[2], a[3], a[4], a[5], a[6], a[7], a[8],
                                     a[9], 1 << 20, None)
        assert st == R.REL_ERR_UNSUPPORTED


def test_linear_gated_validation(lib):
    """The gated Linear Relation entry points need a_log and dt_bias, reject an
    output that overlaps r and a bad RoPE width or base, and take a larger
    backward workspace than the ungated backward (the gate's sums) and a larger
    workspace again with RoPE (its table)."""
    a = ptrs(14)
    p = prob(B=2, H=3, T=300, D=64)
    ws = lib.relation_linear_gated_bwd_workspace_bytes(ctypes.byref(p), 0)
    assert ws > lib.relation_linear_bwd_workspace_bytes(ctypes.byref(p))
    assert lib.relation_linear_gated_bwd_workspace_bytes(ctypes.byref(p), 60) > ws
    fws = lib.relation_linear_gated_fwd_workspace_bytes(ctypes.byref(p), 0)
    assert fws == lib.relation_linear_fwd_workspace_bytes(ctypes.byref(p))
    assert lib.relation_linear_gated_fwd_workspace_bytes(ctypes.byref(p), 64) > fws
    fwd = lambda alog, dtb, rd=0, rb=0.0, pp=p, n=fws: lib.relation_linear_gated_fwd(
        ctypes.byref(pp), a[0], a[1], a[2], a[3], alog, dtb, rd, rb, a[6], None, a[13], n, None)
    assert fwd(a[4], a[5]) == R.REL_ERR_HIP
    assert fwd(None, a[5]) == R.REL_ERR_INVALID_ARG
    assert fwd(a[4], None) == R.REL_ERR_INVALID_ARG
    big = 1 << 22
    assert fwd(a[4], a[5], 60, 1e4, n=big) == R.REL_ERR_HIP       # width 60 of 64
    assert fwd(a[4], a[5], 61, 1e4, n=big) == R.REL_ERR_INVALID_ARG
    assert fwd(a[4], a[5], 66, 1e4, n=big) == R.REL_ERR_INVALID_ARG
    assert fwd(a[4], a[5], 64, 0.0, n=big) == R.REL_ERR_INVALID_ARG
    assert fwd(a[4], a[5], 64, 1e4) == R.REL_ERR_WORKSPACE        # the table does not fit
    p128 = prob(B=1, H=2, T=100, D=128)
    assert fwd(a[4], a[5], 80, 1e4, pp=p128, n=big) == R.REL_ERR_HIP
    assert fwd(a[4], a[5], 60, 1e4, pp=p128, n=big) == R.REL_ERR_UNSUPPORTED
    bwd = lambda dr, rd=0: lib.relation_linear_gated_bwd(ctypes.byref(p), a[0], a[1], a[2], a[3], a[4], a[5], rd,
                                                         1e4, a[6], a[7], a[8], a[9], dr, a[11], a[12], a[13],
                                                         big, None)
    assert bwd(a[10]) == R.REL_ERR_HIP
    assert bwd(a[10], 48) == R.REL_ERR_HIP
    assert bwd(a[3]) == R.REL_ERR_INVALID_ARG  # dr over r
    assert b"overlaps" in lib.relation_last_error()
    st = lib.relation_linear_gated_bwd(ctypes.byref(p), a[0], a[1], a[2], a[3], None, a[5], 0, 0.0, a[6], a[7], a[8],
                                       a[9], a[10], a[11], a[12], a[13], ws, None)
    assert st == R.REL_ERR_INVALID_ARG
