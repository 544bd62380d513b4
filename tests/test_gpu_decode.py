"""GPU parity of the decode step (one new row per (b, h) against a KV cache)
and of its two halves (Exchange scan states of key ranges, and their merge with
the Self entry) against the fp64 decode oracle. fp32: max-abs <= 1e-4; bf16:
relative l2 <= 2e-2."""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

from oracle import decode_oracle as DO
from paper_2608_20172_amd import inputs as I
from paper_2608_20172_amd import binding as R
from tests.gpu_helpers import assert_close, lam_value, log, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    R.load_library()


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _prep(B, H, Tmax, D, dtype, seed, lengths, std=None, lam=0.4):
    inp = I.make_inputs(B, H, Tmax, D, seed=seed, qkv_std=std if std else 1.0 / math.sqrt(D), lam=lam,
                        with_dout=False)
    x = {"lam": lam_value(inp["lam"])}
    x["k"], x["kr"] = to_device(inp["k"], dtype)
    x["v"], x["vr"] = to_device(inp["v"], dtype)
    x["q"], x["qr"] = to_device(inp["q"][:, :, -1], dtype)   # one new query per (b, h)
    x["len"] = torch.tensor(lengths, dtype=torch.int32, device="cuda")
    x["lens"] = list(lengths)
    return x


def _oracle_rows(x, lengths=None):
    B, H, D = x["qr"].shape
    lengths = lengths or x["lens"]
    Y = np.empty((B, H, D))
    M = np.empty((B, H))
    for b in range(B):
        for h in range(H):
            Y[b, h], M[b, h] = DO.decode_step(x["qr"][b, h], x["kr"][b, h], x["vr"][b, h], lengths[b], x["lam"])
    return Y, M


@pytest.mark.parametrize("D,dtype", [(32, "bf16"), (64, "bf16"), (96, "bf16"), (128, "bf16"), (32, "f32"),
                                     (64, "f32"), (128, "f32")])
def test_decode_parity(D, dtype):
    lengths = [1, 2, 333, 700]
    std = 1.0 if dtype == "f32" else None
    x = _prep(4, 3, 700, D, dtype, seed=800 + D, lengths=lengths, std=std)
    log(f"[decode] B=4 H=3 Tmax=700 D={D} {dtype} lengths={lengths}")
    r = R.relation_decode(x["q"], x["k"], x["v"], x["len"], x["lam"])
    torch.cuda.synchronize()
    Y, M = _oracle_rows(x)
    assert_close("y", _np(r["o"]), Y, dtype)
    assert_close("M", _np(r["row_stat"]), M, dtype)
    # one token: y is its own value exactly
    assert np.array_equal(_np(r["o"])[0], x["vr"][0, :, 0])


def test_decode_out_of_range_lengths_give_nan():
    """Cache lengths outside 1..Tmax (0 and Tmax + 1 here) give NaN rows in y
    and M for those batch entries only; the valid entries match the oracle."""
    x = _prep(4, 2, 64, 64, "bf16", seed=810, lengths=[0, 64, 65, 17])
    r = R.relation_decode(x["q"], x["k"], x["v"], x["len"], x["lam"])
    torch.cuda.synchronize()
    o, M = _np(r["o"]), _np(r["row_stat"])
    for b in (0, 2):
        assert np.all(np.isnan(o[b])) and np.all(np.isnan(M[b])), f"entry {b} must be NaN"
    Y, MR = _oracle_rows(x, lengths=[1, 64, 1, 17])
    for b in (1, 3):
        assert_close(f"y[{b}]", o[b], Y[b], "bf16")
        assert_close(f"M[{b}]", M[b], MR[b], "bf16")


def test_decode_is_the_forward_last_row():
    """The decode row of a sequence equals the fused forward's last row."""
    B, H, T, D = 2, 4, 517, 64
    inp = I.make_inputs(B, H, T, D, seed=820, qkv_std=0.125, lam=0.5, with_dout=False)
    q, _ = to_device(inp["q"], "bf16")
    k, kr = to_device(inp["k"], "bf16")
    v, vr = to_device(inp["v"], "bf16")
    lam = lam_value(inp["lam"])
    f = R.relation_fwd(q, k, v, lam)
    r = R.relation_decode(q[:, :, T - 1].contiguous(), k, v, torch.full((B,), T, dtype=torch.int32, device="cuda"),
                          lam)
    torch.cuda.synchronize()
    assert_close("y vs forward", _np(r["o"]), _np(f["o"])[:, :, T - 1], "bf16")
    assert np.max(np.abs(_np(r["row_stat"]) - _np(f["row_stat"])[:, :, T - 1])) < 1e-3


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_decode_states_and_merge(dtype):
    """A cache split in two key ranges (as over two devices): states of each
    range against the oracle's, and their merge against the oracle's row."""
    lengths = [700, 450, 1]
    std = 1.0 if dtype == "f32" else None
    x = _prep(3, 2, 700, 64, dtype, seed=830, lengths=lengths, std=std)
    cut = 300
    s1 = R.relation_decode_states(x["q"], x["k"], x["v"], x["len"], 0, cut, 3)
    s2 = R.relation_decode_states(x["q"], x["k"], x["v"], x["len"], cut, 700, 2)
    r = R.relation_decode_merge(torch.cat([s1, s2]), x["q"], x["k"], x["v"], x["len"], x["lam"])
    torch.cuda.synchronize()
    Y, M = _oracle_rows(x)
    assert_close("merged y", _np(r["o"]), Y, dtype)
    assert_close("merged M", _np(r["row_stat"]), M, dtype)
    # each slice's state against the oracle's state of the same keys
    st = np.concatenate([_np(s1), _np(s2)])
    bounds = [(0, 100), (100, 200), (200, 300), (300, 500), (500, 700)]
    for si, (k0, k1) in enumerate(bounds):
        for n in range(6):
            b, h = divmod(n, 2)
            keys = np.arange(k0, min(k1, lengths[b] - 1))
            m, l, z = DO.exchange_state(x["qr"][b, h], x["kr"][b, h], x["vr"][b, h], keys)
            gm, gl, gz = st[si, n, 0], st[si, n, 1], st[si, n, 2:]
            if keys.size == 0:
                assert gm == -np.inf and gl == 0.0 and not gz.any(), (si, n)
                continue
            assert abs(gm - m) <= 1e-4 * max(1.0, abs(m)), (si, n, gm, m)
            assert abs(gl - l) <= 1e-4 * l, (si, n, gl, l)
            assert np.max(np.abs(gz - z)) <= 1e-4 * max(1.0, np.max(np.abs(z))), (si, n)
    # no states at all: every row is pure Self
    r0 = R.relation_decode_merge(torch.empty((0, 6, 66), device="cuda"), x["q"], x["k"], x["v"], x["len"], x["lam"])
    torch.cuda.synchronize()
    for b, L in enumerate(lengths):
        assert np.array_equal(_np(r0["o"])[b], x["vr"][b, :, L - 1])


def test_decode_long_context():
    """One sequence of 16384 tokens, 16 heads of width 128: every head against the oracle."""
    x = _prep(1, 16, 16384, 128, "bf16", seed=840, lengths=[16384])
    r = R.relation_decode(x["q"], x["k"], x["v"], x["len"], x["lam"])
    torch.cuda.synchronize()
    Y, M = _oracle_rows(x)
    assert_close("y", _np(r["o"]), Y, "bf16")
    assert_close("M", _np(r["row_stat"]), M, "bf16")


def test_decode_repeatable():
    x = _prep(4, 12, 2048, 64, "bf16", seed=850, lengths=[2048, 1500, 700, 2])
    a = R.relation_decode(x["q"], x["k"], x["v"], x["len"], x["lam"])
    b = R.relation_decode(x["q"], x["k"], x["v"], x["len"], x["lam"])
    torch.cuda.synchronize()
    assert torch.equal(a["o"], b["o"]) and torch.equal(a["row_stat"], b["row_stat"])
