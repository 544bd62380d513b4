"""relation_bwd_noalloc (its scratch in the library's own per-device array, no
allocation inside the call) against relation_bwd on the same inputs: two calls
in a row, the second on a smaller problem, so the second call runs on scratch
the first one left behind."""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

from paper_2608_20172_amd import binding as R
from paper_2608_20172_amd import inputs as I
from tests.gpu_helpers import assert_close, assert_scalar_close, lam_value, log, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    R.load_library()


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


CASES = [  # (B, H, T, D, dtype, seed): the second call is smaller than the first
    (2, 3, 700, 64, "bf16", 81),
    (1, 2, 150, 64, "bf16", 82),
    (1, 2, 190, 32, "f32", 83),
    (1, 1, 65, 128, "bf16", 84),
]


def test_noalloc_backward_matches_relation_bwd():
    lib = R.load_library()
    assert lib.relation_bwd_noalloc_max_scratch_bytes() == 32 << 20
    for (B, H, T, D, dtype, seed) in CASES:
        log(f"[noalloc] B={B} H={H} T={T} D={D} {dtype} seed={seed}")
        inp = I.make_inputs(B, H, T, D, seed=seed, qkv_std=1 / math.sqrt(D) if dtype == "bf16" else 1.0, lam=0.4)
        q, _ = to_device(inp["q"], dtype)
        k, _ = to_device(inp["k"], dtype)
        v, _ = to_device(inp["v"], dtype)
        do, _ = to_device(inp["dout"], dtype)
        lam = torch.tensor([lam_value(inp["lam"])], dtype=torch.float32, device="cuda")
        f = R.relation_fwd(q, k, v, lam)
        ref = R.relation_bwd(q, k, v, f["o"], do, lam, f["row_stat"], want_dself=True)
        got = R.relation_bwd_noalloc(q, k, v, f["o"], do, lam, f["row_stat"], want_dself=True)
        torch.cuda.synchronize()
        for n in ("dq", "dk", "dv", "dself"):
            assert_close(f"noalloc {n}", _np(got[n]), _np(ref[n]), dtype)
        i1 = np.log(np.arange(1, T + 1, dtype=np.float64))
        assert_scalar_close("noalloc dlambda", float(got["dlambda"].item()), float(ref["dlambda"].item()),
                            i1[None, None, :] * _np(ref["dself"]), dtype)
