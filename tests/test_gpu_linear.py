"""GPU parity of Linear Relation (the recurrent-state Exchange) against the
fp64 oracle's token-by-token recurrence, on the same seeded inputs. fp32:
max-abs <= 1e-4; bf16: relative l2 <= 2e-2."""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

from oracle import linear_oracle as LO
from paper_2608_20172_amd import inputs as I
from paper_2608_20172_amd import binding as R
from tests.gpu_helpers import assert_close, log, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    R.load_library()


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _prep(B, H, T, D, dtype, seed, gmax=0.5, with_dout=True):
    inp = I.make_inputs(B, H, T, D, seed=seed, qkv_std=1.0, with_dout=with_dout)
    x = {}
    for n, src in (("p1", "q"), ("p2", "k"), ("v", "v")):
        x[n], x[n + "r"] = to_device(inp[src], dtype)
    if with_dout:
        x["dy"], x["dyr"] = to_device(inp["dout"], dtype)
    g = np.asarray(I.make_log_retention(B, H, T, D, seed=seed, gmax=gmax), dtype=np.float32)
    x["g"] = torch.from_numpy(g).cuda()
    x["gr"] = g.astype(np.float64)
    return x


def check_linear_fwd(x, dtype, heads=None):
    B, H, T, D = x["p1"].shape
    log(f"[linear fwd] B={B} H={H} T={T} D={D} {dtype}")
    r = R.relation_linear_fwd(x["p1"], x["p2"], x["v"], x["g"], want_state=True)
    torch.cuda.synchronize()
    heads = heads or [(b, h) for b in range(B) for h in range(H)]
    for b, h in heads:
        f = LO.forward(x["p1r"][b, h], x["p2r"][b, h], x["vr"][b, h], x["gr"][b, h])
        assert_close(f"y[{b},{h}]", _np(r["o"])[b, h], f["Y"], dtype)
        assert_close(f"state[{b},{h}]", _np(r["state"])[b, h], f["C"], dtype)
    return r


@pytest.mark.parametrize("B,H,T,D,dtype", [
    (2, 2, 300, 64, "bf16"), (1, 2, 190, 32, "f32"), (1, 2, 200, 128, "bf16"), (1, 3, 64, 64, "f32"),
    (1, 2, 1, 64, "bf16"), (1, 2, 65, 64, "bf16"), (1, 2, 129, 128, "f32"),
])
def test_linear_forward(B, H, T, D, dtype):
    x = _prep(B, H, T, D, dtype, seed=1000 + T + D)
    r = check_linear_fwd(x, dtype)
    if T == 1:
        assert np.array_equal(_np(r["o"]), x["vr"])


@pytest.mark.parametrize("gmax", [1e-3, 8.0, 80.0])
def test_linear_forward_retention_range(gmax):
    """Long memory (alpha near 1), fast forgetting, and retention that
    underflows to zero within a chunk."""
    x = _prep(1, 2, 257, 64, "f32", seed=1100, gmax=gmax)
    check_linear_fwd(x, "f32")


def test_linear_forward_long():
    x = _prep(1, 4, 2048, 64, "bf16", seed=1200, gmax=0.05)
    check_linear_fwd(x, "bf16", heads=[(0, 0), (0, 3)])


@pytest.mark.parametrize("T,gmax", [(1024, 0.02), (1025, 0.02), (3000, 0.005), (3000, 2.0)])
def test_linear_forward_scan_segments(T, gmax):
    """The state scan works over segments of 16 chunks (1024 tokens): one full
    segment, one plus a one-token chunk, and three with a ragged last chunk,
    with slow retention so that the state crosses segment boundaries."""
    x = _prep(1, 2, T, 64, "f32", seed=1250 + T, gmax=gmax)
    check_linear_fwd(x, "f32")


def test_linear_forward_strided():
    x = _prep(2, 3, 150, 64, "bf16", seed=1300)
    a = R.relation_linear_fwd(x["p1"], x["p2"], x["v"], x["g"])
    t = lambda z: z.transpose(1, 2).contiguous().transpose(1, 2)
    b = R.relation_linear_fwd(t(x["p1"]), t(x["p2"]), t(x["v"]), x["g"])
    torch.cuda.synchronize()
    assert torch.equal(a["o"], b["o"].contiguous())


def check_linear_bwd(x, dtype, heads=None):
    B, H, T, D = x["p1"].shape
    log(f"[linear bwd] B={B} H={H} T={T} D={D} {dtype}")
    r = R.relation_linear_bwd(x["p1"], x["p2"], x["v"], x["g"], x["dy"])
    torch.cuda.synchronize()
    heads = heads or [(b, h) for b in range(B) for h in range(H)]
    for b, h in heads:
        o = LO.backward(x["p1r"][b, h], x["p2r"][b, h], x["vr"][b, h], x["gr"][b, h], x["dyr"][b, h])
        for n in ("dp1", "dp2", "dv", "dg"):
            assert_close(f"{n}[{b},{h}]", _np(r[n])[b, h], o[n], dtype)
    return r


@pytest.mark.parametrize("B,H,T,D,dtype", [
    (2, 2, 300, 64, "bf16"), (1, 2, 190, 32, "f32"), (1, 3, 64, 64, "f32"), (1, 2, 1, 64, "bf16"),
    (1, 2, 65, 32, "bf16"), (1, 2, 129, 64, "f32"),
    # width 128: four 64-channel problems per head, summed
    (1, 2, 200, 128, "bf16"), (2, 2, 129, 128, "f32"), (1, 1, 1, 128, "bf16"), (1, 3, 64, 128, "f32"),
])
def test_linear_backward(B, H, T, D, dtype):
    x = _prep(B, H, T, D, dtype, seed=1400 + T + D)
    check_linear_bwd(x, dtype)


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("gmax", [1e-3, 8.0, 80.0])
def test_linear_backward_retention_range(gmax, D):
    x = _prep(1, 2, 200, D, "f32", seed=1500 + D, gmax=gmax)
    check_linear_bwd(x, "f32")


@pytest.mark.parametrize("D,gmax", [(64, 1e-3), (64, 8.0), (64, 80.0), (128, 80.0)])
def test_linear_backward_retention_range_bf16(D, gmax):
    """The same retention range with bf16 inputs, where the chunk products
    take bf16 operands: decay factors down to underflow inside the operands."""
    x = _prep(1, 2, 200, D, "bf16", seed=1550 + D, gmax=gmax)
    check_linear_fwd(x, "bf16")
    check_linear_bwd(x, "bf16")


def test_linear_backward_long():
    x = _prep(1, 2, 2048, 64, "bf16", seed=1600, gmax=0.05)
    check_linear_bwd(x, "bf16", heads=[(0, 1)])


@pytest.mark.parametrize("T,D,gmax", [(1025, 64, 0.02), (3000, 64, 0.005), (2100, 32, 0.01), (2100, 128, 0.01)])
def test_linear_backward_scan_segments(T, D, gmax):
    """Forward and reverse state scans across segments of 16 chunks."""
    x = _prep(1, 1, T, D, "f32", seed=1650 + T + D, gmax=gmax)
    check_linear_bwd(x, "f32")


@pytest.mark.parametrize("D", [64, 128])
def test_linear_backward_strided(D):
    """Token-major tensors (strides of a [B, T, H, D] layout) give the same
    gradients as contiguous ones."""
    x = _prep(2, 3, 150, D, "bf16", seed=1680 + D)
    a = R.relation_linear_bwd(x["p1"], x["p2"], x["v"], x["g"], x["dy"])
    t = lambda z: z.transpose(1, 2).contiguous().transpose(1, 2)
    b = R.relation_linear_bwd(t(x["p1"]), t(x["p2"]), t(x["v"]), x["g"], t(x["dy"]))
    torch.cuda.synchronize()
    for n in ("dp1", "dp2", "dv", "dg"):
        assert torch.equal(a[n].contiguous(), b[n].contiguous()), n


def _misaligned(t):
    """The same values in a view that starts one element past a 16-byte boundary."""
    buf = torch.empty(t.numel() + 1, dtype=t.dtype, device=t.device)
    v = buf[1:].view(t.shape)
    v.copy_(t)
    return v


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_linear_unaligned_rows(dtype, D):
    """Rows that do not start on 16-byte boundaries take the element-wise chunk
    loads; forward and backward against the oracle."""
    x = _prep(1, 2, 200, D, dtype, seed=1690 + D)
    for n in ("p1", "p2", "v", "dy", "g"):
        x[n] = _misaligned(x[n])
    check_linear_fwd(x, dtype)
    check_linear_bwd(x, dtype)


@pytest.mark.parametrize("D", [64, 128])
def test_linear_backward_repeatable(D):
    x = _prep(2, 2, 300, D, "bf16", seed=1700 + D)
    a = R.relation_linear_bwd(x["p1"], x["p2"], x["v"], x["g"], x["dy"])
    b = R.relation_linear_bwd(x["p1"], x["p2"], x["v"], x["g"], x["dy"])
    torch.cuda.synchronize()
    for n in ("dp1", "dp2", "dv", "dg"):
        assert torch.equal(a[n], b[n]), n


def _pad(t, width):
    return torch.nn.functional.pad(t, (0, width - t.shape[-1]))


@pytest.mark.parametrize("width,padded,T,dtype", [(80, 128, 300, "bf16"), (80, 128, 130, "f32"),
                                                   (48, 64, 200, "bf16"), (60, 64, 129, "f32")])
def test_linear_padded_head_width(width, padded, T, dtype):
    """The paper's head widths (48, 60, 80) run zero-padded to a supported one
    with the scale of the true width: p1, p2, v, dY and g padded with zeros
    (alpha = 1 on the padded channels, whose state rows and columns stay
    zero). y and every gradient match the oracle at the true width on the
    first channels and are zero on the padding."""
    x = _prep(1, 2, T, width, dtype, seed=1800 + width + T)
    pad = {n: _pad(x[n], padded).contiguous() for n in ("p1", "p2", "v", "dy", "g")}
    scale = 1.0 / math.sqrt(width)
    log(f"[linear padded] width {width} -> {padded}, T={T} {dtype}")
    f = R.relation_linear_fwd(pad["p1"], pad["p2"], pad["v"], pad["g"], scale=scale)
    r = R.relation_linear_bwd(pad["p1"], pad["p2"], pad["v"], pad["g"], pad["dy"], scale=scale)
    torch.cuda.synchronize()
    for h in range(2):
        ref_f = LO.forward(x["p1r"][0, h], x["p2r"][0, h], x["vr"][0, h], x["gr"][0, h])
        ref_b = LO.backward(x["p1r"][0, h], x["p2r"][0, h], x["vr"][0, h], x["gr"][0, h], x["dyr"][0, h])
        y = _np(f["o"])[0, h]
        assert_close(f"y[0,{h}]", y[:, :width], ref_f["Y"], dtype)
        assert not np.any(y[:, width:])
        for n in ("dp1", "dp2", "dv", "dg"):
            got = _np(r[n])[0, h]
            assert_close(f"{n}[0,{h}]", got[:, :width], ref_b[n], dtype)
            assert not np.any(got[:, width:]), f"{n}: padding channels non-zero"


def _gate_params(H, D, seed, a_mean=0.0):
    rng = np.random.default_rng(seed + 7919)
    a_log = (a_mean + 0.5 * rng.standard_normal((H, D))).astype(np.float32)
    dt_bias = rng.standard_normal((H, D)).astype(np.float32)
    return a_log, dt_bias


def _assert_param_grad(name, x, ref, terms, dtype):
    """A per-(head, channel) sum over batch entries and tokens: each entry's
    error against the bar times the larger of |ref| and the l2 norm of its
    terms (bf16), or max-abs against the larger of 1e-4 and 1e-5 of the sum of
    |terms| (fp32)."""
    err = np.abs(np.asarray(x, np.float64) - ref)
    t = np.abs(terms)
    if dtype == "f32":
        lim = np.maximum(1e-4, 1e-5 * t.sum(axis=(0, 2)))
    else:
        lim = 2e-2 * np.maximum(np.abs(ref), np.sqrt(np.sum(t * t, axis=(0, 2))))
    zero = lim == 0.0  # no terms (T = 1 has no history): the sum must be zero
    assert np.all(err[zero] == 0.0), f"{name}: non-zero where every term is zero"
    worst = float(np.max(err[~zero] / lim[~zero])) if np.any(~zero) else 0.0
    log(f"  {name}: worst error / allowance {worst:.3e}")
    assert worst <= 1.0, f"{name}: error {worst:.3e} of the allowance"


@pytest.mark.parametrize("B,H,T,D,dtype,a_mean", [
    (2, 2, 300, 64, "bf16", 0.0), (1, 2, 190, 32, "f32", 0.0), (1, 2, 200, 128, "bf16", 0.0),
    (2, 1, 129, 128, "f32", -1.0), (1, 2, 1, 64, "bf16", 0.0), (1, 1, 600, 64, "f32", -4.0),
    # long sequences: dA_log and d dt_bias sum over every token, so an error in
    # dg that is coherent over the tokens would outgrow the allowance here
    (1, 2, 8192, 64, "bf16", 0.0), (1, 1, 2048, 128, "bf16", 0.0),
])
def test_linear_gated(B, H, T, D, dtype, a_mean):
    """The retention gate of eq. 15 formed in the kernels: y and the state, then
    dp1, dp2, dv, dr and the per-channel dA_log, d dt_bias, against the oracle's
    gate composed with its recurrence (the gate's adjoint fed the recurrence's
    dg)."""
    x = _prep(B, H, T, D, dtype, seed=1900 + T + D, with_dout=True)
    rng = np.random.default_rng(1950 + T)
    r = (2.0 * rng.standard_normal((B, H, T, D))).astype(np.float32)
    a_log, dt_bias = _gate_params(H, D, 1960 + T, a_mean)
    rt, at, bt = (torch.from_numpy(z).cuda() for z in (r, a_log, dt_bias))
    log(f"[linear gated] B={B} H={H} T={T} D={D} {dtype} A_log mean {a_mean}")
    f = R.relation_linear_gated_fwd(x["p1"], x["p2"], x["v"], rt, at, bt, want_state=True)
    o = R.relation_linear_gated_bwd(x["p1"], x["p2"], x["v"], rt, at, bt, x["dy"])
    torch.cuda.synchronize()
    da_terms = np.zeros((B, H, T, D))
    dt_terms = np.zeros((B, H, T, D))
    da_ref = np.zeros((H, D))
    dt_ref = np.zeros((H, D))
    for b in range(B):
        for h in range(H):
            g = LO.kda_gate(r[b, h], a_log[h], dt_bias[h])
            ref_f = LO.forward(x["p1r"][b, h], x["p2r"][b, h], x["vr"][b, h], g)
            assert_close(f"y[{b},{h}]", _np(f["o"])[b, h], ref_f["Y"], dtype)
            assert_close(f"state[{b},{h}]", _np(f["state"])[b, h], ref_f["C"], dtype)
            ref_b = LO.backward(x["p1r"][b, h], x["p2r"][b, h], x["vr"][b, h], g, x["dyr"][b, h])
            gb = LO.kda_gate_backward(r[b, h], a_log[h], dt_bias[h], ref_b["dg"])
            for n in ("dp1", "dp2", "dv"):
                assert_close(f"{n}[{b},{h}]", _np(o[n])[b, h], ref_b[n], dtype)
            assert_close(f"dr[{b},{h}]", _np(o["dr"])[b, h], gb["dr"], dtype)
            da_terms[b, h] = ref_b["dg"] * g
            dt_terms[b, h] = gb["dr"]
            da_ref[h] += gb["da_log"]
            dt_ref[h] += gb["ddt_bias"]
    _assert_param_grad("da_log", _np(o["da_log"]), da_ref, da_terms, dtype)
    _assert_param_grad("ddt_bias", _np(o["ddt_bias"]), dt_ref, dt_terms, dtype)


def test_linear_gated_unaligned_params():
    """A_log and dt_bias at addresses that are not 16-byte aligned (views one
    element into a buffer) take the element-wise chunk loads; y, the state and
    every gradient agree with the oracle as with aligned parameters."""
    B, H, T, D = 1, 2, 150, 64
    x = _prep(B, H, T, D, "bf16", seed=1970, with_dout=True)
    rng = np.random.default_rng(1971)
    r = (2.0 * rng.standard_normal((B, H, T, D))).astype(np.float32)
    a_log, dt_bias = _gate_params(H, D, 1972)
    rt = torch.from_numpy(r).cuda()
    abuf = torch.zeros(H * D + 1, dtype=torch.float32, device="cuda")
    bbuf = torch.zeros(H * D + 1, dtype=torch.float32, device="cuda")
    abuf[1:] = torch.from_numpy(a_log.ravel()).cuda()
    bbuf[1:] = torch.from_numpy(dt_bias.ravel()).cuda()
    at, bt = abuf[1:].view(H, D), bbuf[1:].view(H, D)
    assert at.data_ptr() % 16 and bt.data_ptr() % 16
    f = R.relation_linear_gated_fwd(x["p1"], x["p2"], x["v"], rt, at, bt, want_state=True)
    o = R.relation_linear_gated_bwd(x["p1"], x["p2"], x["v"], rt, at, bt, x["dy"])
    torch.cuda.synchronize()
    for h in range(H):
        g = LO.kda_gate(r[0, h], a_log[h], dt_bias[h])
        ref_f = LO.forward(x["p1r"][0, h], x["p2r"][0, h], x["vr"][0, h], g)
        assert_close(f"y[0,{h}]", _np(f["o"])[0, h], ref_f["Y"], "bf16")
        ref_b = LO.backward(x["p1r"][0, h], x["p2r"][0, h], x["vr"][0, h], g, x["dyr"][0, h])
        gb = LO.kda_gate_backward(r[0, h], a_log[h], dt_bias[h], ref_b["dg"])
        for n in ("dp1", "dp2", "dv"):
            assert_close(f"{n}[0,{h}]", _np(o[n])[0, h], ref_b[n], "bf16")
        assert_close(f"dr[0,{h}]", _np(o["dr"])[0, h], gb["dr"], "bf16")


def test_linear_gated_repeatable():
    x = _prep(2, 2, 700, 64, "bf16", seed=1990)
    rng = np.random.default_rng(1991)
    r = torch.from_numpy(rng.standard_normal((2, 2, 700, 64)).astype(np.float32)).cuda()
    a_log, dt_bias = (torch.from_numpy(z).cuda() for z in _gate_params(2, 64, 1992))
    a = R.relation_linear_gated_bwd(x["p1"], x["p2"], x["v"], r, a_log, dt_bias, x["dy"])
    b = R.relation_linear_gated_bwd(x["p1"], x["p2"], x["v"], r, a_log, dt_bias, x["dy"])
    torch.cuda.synchronize()
    for n in ("dp1", "dp2", "dv", "dr", "da_log", "ddt_bias"):
        assert torch.equal(a[n], b[n]), n


@pytest.mark.parametrize("D,dtype", [(64, "f32"), (32, "bf16"), (128, "f32")])
def test_linear_mixed_decay_chunks(D, dtype):
    """Chunks whose decay inside a 16-token block is mild take the factored
    diagonal blocks on the matrix cores, chunks with steep decay (here up to
    e^-20 per token) the term-by-term path; one sequence with both kinds,
    forward and backward against the oracle."""
    T = 64 * 5 + 17
    x = _prep(1, 2, T, D, dtype, seed=2100 + D)
    rng = np.random.default_rng(2101)
    gmax = np.where((np.arange(T) // 64) % 2 == 1, 20.0, 0.05)[None, None, :, None]
    g = (-rng.uniform(0.0, 1.0, (1, 2, T, D)) * gmax).astype(np.float32)
    x["g"] = torch.from_numpy(g).cuda()
    x["gr"] = g.astype(np.float64)
    check_linear_fwd(x, dtype)
    check_linear_bwd(x, dtype)


@pytest.mark.parametrize("width,padded,T,dtype", [(64, 64, 300, "bf16"), (32, 32, 190, "f32"), (128, 128, 200, "bf16"),
                                                   (80, 128, 260, "f32"), (60, 64, 129, "f32"), (48, 64, 200, "bf16"),
                                                   (80, 128, 300, "bf16")])
def test_linear_gated_rope(width, padded, T, dtype):
    """RoPE (base 1e4) on p1, p2 inside the gated kernels, over the true width
    of a head zero-padded to a kernel width: y, dp1, dp2, dv, dr, dA_log and
    d dt_bias against the oracle's RoPE (the layer oracle's rotate-half)
    composed with the gate and the recurrence at the true width, and zeros on
    the padding."""
    from oracle import layer_oracle as LR
    B, H = 1, 2
    x = _prep(B, H, T, width, dtype, seed=2200 + width + T)
    rng = np.random.default_rng(2201 + T)
    r = (2.0 * rng.standard_normal((B, H, T, width))).astype(np.float32)
    a_log, dt_bias = _gate_params(H, width, 2202 + T)
    pad = {n: _pad(x[n], padded).contiguous() for n in ("p1", "p2", "v", "dy")}
    rt = _pad(torch.from_numpy(r), padded).contiguous().cuda()
    at, bt = (_pad(torch.from_numpy(z), padded).contiguous().cuda() for z in (a_log, dt_bias))
    scale = 1.0 / math.sqrt(width)
    log(f"[linear gated rope] width {width} -> {padded}, T={T} {dtype}")
    f = R.relation_linear_gated_fwd(pad["p1"], pad["p2"], pad["v"], rt, at, bt, rope_dim=width, rope_base=1e4,
                                    scale=scale)
    o = R.relation_linear_gated_bwd(pad["p1"], pad["p2"], pad["v"], rt, at, bt, pad["dy"], rope_dim=width,
                                    rope_base=1e4, scale=scale)
    torch.cuda.synchronize()
    da_ref, dt_ref = np.zeros((H, width)), np.zeros((H, width))
    da_terms, dt_terms = np.zeros((B, H, T, width)), np.zeros((B, H, T, width))
    for h in range(H):
        p1r, p2r = LR.rope(x["p1r"][0, h], 1e4), LR.rope(x["p2r"][0, h], 1e4)
        g = LO.kda_gate(r[0, h], a_log[h], dt_bias[h])
        ref_f = LO.forward(p1r, p2r, x["vr"][0, h], g)
        y = _np(f["o"])[0, h]
        assert_close(f"y[0,{h}]", y[:, :width], ref_f["Y"], dtype)
        assert not np.any(y[:, width:])
        ref_b = LO.backward(p1r, p2r, x["vr"][0, h], g, x["dyr"][0, h])
        gb = LO.kda_gate_backward(r[0, h], a_log[h], dt_bias[h], ref_b["dg"])
        want = {"dp1": LR.rope_transpose(ref_b["dp1"], 1e4), "dp2": LR.rope_transpose(ref_b["dp2"], 1e4),
                "dv": ref_b["dv"], "dr": gb["dr"]}
        for n, ref in want.items():
            got = _np(o[n])[0, h]
            assert_close(f"{n}[0,{h}]", got[:, :width], ref, dtype)
            assert not np.any(got[:, width:]), f"{n}: padding channels non-zero"
        da_ref[h], dt_ref[h] = gb["da_log"], gb["ddt_bias"]
        da_terms[0, h], dt_terms[0, h] = ref_b["dg"] * g, gb["dr"]
    _assert_param_grad("da_log", _np(o["da_log"])[:, :width], da_ref, da_terms, dtype)
    _assert_param_grad("ddt_bias", _np(o["ddt_bias"])[:, :width], dt_ref, dt_terms, dtype)
