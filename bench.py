#!/usr/bin/env python3
"""Benchmark of the fused causal Full Relation operator (FlashRelation) on one
MI355X: forward + backward tokens/s on the 100M-decoder-scale layer
(B=8, H=12, T=2048, D=64, bf16, 5% of query rows boosted x8).

One step = relation_fwd + relation_bwd over the whole batch, inputs resident
in HBM. Prints one JSON line. Extra legs: the materialised baseline's forward
and backward (for the speedups), per-kernel durations from HIP events
recorded around the fused kernels inside the timed region, the measured MFMA
peak, the other decoder-scale and long-context workloads, the layer entry
points at the paper's 100M geometry, decode steps, Linear Relation, and the
fp64 oracle on a bounded sample of heads on the host cores.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
  python bench.py --copy-bytes N   # plain device copy of N bytes (counter calibration)
  python bench.py --summarize-counters F.csv W.csv CF.csv CW.csv --copy-bytes N
                                   # backward HBM traffic from rocprofv3 --pmc runs
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2608_20172_amd.inputs import WORKLOADS, make_workload_inputs  # noqa: E402

METRIC = "FlashRelation fwd+bwd tokens/s and % bf16 MFMA peak; speedup vs materialised"
PEAK_BF16 = 2.5e15      # MI355X dense bf16 MFMA, FLOP/s
PEAK_HBM = 8.0e12       # MI355X HBM3E, B/s
MATERIALIZED_BUDGET = 8 << 30  # bytes of T x T workspace the baseline may use
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "bwd_kernel_traffic.json")
KERNEL_SOURCES = ["paper_2608_20172_amd/csrc/bwd.hip", "paper_2608_20172_amd/csrc/common.h"]


def pairs(T: int) -> int:
    return T * (T - 1) // 2


def flops(w, which: str) -> float:
    """Algorithmic MFMA flops: forward 4 D per strictly causal pair (QK^T and
    F V), backward 10 D (QK^T recomputed, dO V^T, F^T dO, dU^T Q, dU K)."""
    per = {"fwd": 4, "bwd": 10}[which]
    return float(per * w.D * w.N * pairs(w.T))


def sources_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


# ---------------------------------------------------------------------------
# CPU baseline: the fp64 oracle on a bounded sample of heads
# ---------------------------------------------------------------------------
def _warm_worker(_):
    import oracle  # noqa: F401
    import scipy.special  # noqa: F401
    from threadpoolctl import threadpool_limits  # noqa: F401
    return os.getpid()


def _oracle_head(args):
    q, k, v, do, lam = args
    from threadpoolctl import threadpool_limits
    import oracle
    with threadpool_limits(1):
        t0 = time.perf_counter()
        oracle.forward(q, k, v, lam, want_matrices=False, row_block=256)
        oracle.backward(q, k, v, lam, do, row_block=256)
        return time.perf_counter() - t0


def cpu_baseline(w, rounded, lam, budget_s: float) -> dict:
    import multiprocessing as mp
    import numpy as np
    workers = max(1, min(16, os.cpu_count() or 1))
    heads = [(b, h) for b in range(w.B) for h in range(w.H)]
    # one head to size the sample, then enough heads for ~budget_s of CPU work
    probe = _oracle_head((rounded["q"][0, 0], rounded["k"][0, 0], rounded["v"][0, 0],
                          rounded["dout"][0, 0], lam))
    n = int(max(workers, min(len(heads), round(budget_s / max(probe, 1e-3)))))
    n = max(1, min(len(heads), (n // workers) * workers or workers))
    sample = heads[:n]
    jobs = [(rounded["q"][b, h], rounded["k"][b, h], rounded["v"][b, h], rounded["dout"][b, h], lam)
            for (b, h) in sample]
    ctx = mp.get_context("spawn")
    with ctx.Pool(workers) as pool:
        pool.map(_warm_worker, range(4 * workers))  # start-up and imports are not timed
        t0 = time.perf_counter()
        per_head = pool.map(_oracle_head, jobs, chunksize=1)
        wall = time.perf_counter() - t0
    full_wall = wall * len(heads) / len(sample)
    return {
        "value": w.tokens / full_wall,
        "unit": "tokens/s",
        "cores": workers,
        "kind": "oracle",
        "sample": (f"fp64 oracle forward+backward on {len(sample)} of {len(heads)} heads "
                   f"(T={w.T}, D={w.D}), {workers} worker processes x 1 BLAS thread, "
                   f"{wall:.1f} s wall / {sum(per_head):.1f} s CPU; scaled to all heads"),
    }


def round_inputs(inp, dtype: str) -> dict:
    """The exact values the device receives, as fp64 (bf16 rounding by torch on the CPU)."""
    import torch
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    out = {}
    for n in ("q", "k", "v", "dout"):
        if inp.get(n) is not None:
            out[n] = torch.from_numpy(inp[n]).to(tdt).to(torch.float64).numpy()
    return out


# ---------------------------------------------------------------------------
# HIP events through the runtime library (recorded by librelation itself)
# ---------------------------------------------------------------------------
class Hip:
    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def events(self, n):
        evs = []
        for _ in range(n):
            e = ctypes.c_void_p()
            if self.lib.hipEventCreate(ctypes.byref(e)) != 0:
                raise RuntimeError("hipEventCreate failed")
            evs.append(e.value)
        return evs

    def elapsed_ms(self, a, b) -> float:
        ms = ctypes.c_float()
        if self.lib.hipEventElapsedTime(ctypes.byref(ms), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def destroy(self, evs):
        for e in evs:
            self.lib.hipEventDestroy(e)


def arm(lib, kernel: str, evs):
    arr = (ctypes.c_void_p * len(evs))(*evs)
    st = lib.relation_profile_arm(kernel.encode(), arr, len(evs) // 2)
    if st != 0:
        raise RuntimeError("relation_profile_arm failed")
    return arr


def traffic_for(kernel_hash: str, kernel=None):
    """HBM bytes per launch of one kernel of the backward (``kernel``: its key
    in the summary's per_kernel table), or of the whole one-kernel backward,
    from the committed counter summary, if it was taken on the current kernel
    source."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("sources_hash") != kernel_hash:
        return None
    if kernel is not None:
        return t.get("per_kernel", {}).get(kernel, {}).get("bytes")
    return t.get("bytes_per_launch")


def _counter_rows(path: str) -> dict:
    """Mean counter value per kernel over the dispatches of a rocprofv3
    --pmc CSV (one row per dispatch and counter; repeated rows of one
    dispatch are collapsed)."""
    import csv
    seen, acc = set(), {}
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            key = (r["Dispatch_Id"], r["Counter_Name"])
            if key in seen:
                continue
            seen.add(key)
            acc.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in acc.items()}


# kernels of the 100M-scale layer's step (bf16, D = 64), by the parts of their names
STEP_KERNELS = {
    "fwd_kernel": ("fwd_kernel<", "PolBF16<64>"),
    "bwd_prep_kernel": ("bwd_prep_kernel<64>",),
    "bwd_fused_kernel": ("bwd_dkdv_kernel<", "PolBF16<64>", "8, true"),
    "bwd_dq_convert_kernel": ("bwd_dq_convert_kernel<64>",),
    "bwd_dq_kernel": ("bwd_dq_kernel<", "PolBF16<64>"),
    "bwd_dkdv_kernel": ("bwd_dkdv_kernel<", "PolBF16<64>", "4, false"),
}
ONE_KERNEL_BWD = ("bwd_prep_kernel", "bwd_fused_kernel", "bwd_dq_convert_kernel")
TWO_KERNEL_BWD = ("bwd_dq_kernel", "bwd_dkdv_kernel")


def summarize_counters(paths, copy_bytes: int) -> dict:
    """HBM bytes per launch of each kernel of the step from FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch), each scaled by what the same counter reads
    for a plain device copy of ``copy_bytes`` bytes (read once, written once)."""
    fetch, write, cfetch, cwrite = (_counter_rows(p) for p in paths)
    copy_name = max(cfetch, key=cfetch.get)
    f_scale = copy_bytes / (cfetch[copy_name] * 1024.0)
    w_scale = copy_bytes / (cwrite[max(cwrite, key=cwrite.get)] * 1024.0)
    per = {}
    for short, parts in STEP_KERNELS.items():
        names = [n for n in fetch if all(x in n for x in parts)]
        if not names:
            continue
        n = names[0]
        fb = fetch[n] * 1024.0 * f_scale
        wb = write.get(n, 0.0) * 1024.0 * w_scale
        per[short] = {"name": n, "fetch_kib_raw": fetch[n], "write_kib_raw": write.get(n, 0.0),
                      "read_bytes": fb, "write_bytes": wb, "bytes": fb + wb}
    one = sum(per[k]["bytes"] for k in ONE_KERNEL_BWD) if all(k in per for k in ONE_KERNEL_BWD) else None
    two = sum(per[k]["bytes"] for k in TWO_KERNEL_BWD) if all(k in per for k in TWO_KERNEL_BWD) else None
    return {"sources_hash": sources_hash(), "workload": "dec100m_T2048",
            "bytes_per_launch": one, "bytes_per_launch_two_kernel": two, "per_kernel": per,
            "calibration": {"copy_bytes": copy_bytes, "copy_kernel": copy_name,
                            "fetch_factor": f_scale, "write_factor": w_scale}}


# ---------------------------------------------------------------------------
def copy_mode(nbytes: int, reps: int, kind: str) -> None:
    """A plain device copy of nbytes (read once, written once), for scaling
    the memory counters: 'memcpy' is the runtime's copy kernel, 'elementwise'
    a vectorised elementwise kernel (16-byte loads per lane, like the fused
    kernels)."""
    import torch
    x = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").uniform_()
    y = torch.empty_like(x)
    for _ in range(reps):
        if kind == "memcpy":
            y.copy_(x)
        else:
            torch.mul(x, 1.0, out=y)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "reps": reps, "kind": kind}), flush=True)


def materialized_backward(w, q, k, v, do, lam_t, fwd_ms, bwd_ms, mat_fwd_ms, K, args):
    """Time the materialised backward (U and H = dO V^T in HBM, dU and F written
    for the three gradient GEMMs) and compare whole steps."""
    import torch
    from paper_2608_20172_amd import binding as R
    need = R.relation_bwd_materialized_workspace_bytes(q)
    if need > MATERIALIZED_BUDGET:
        return {"bwd_status": f"skipped: T x T workspace {need / 2**30:.1f} GiB exceeds the "
                              f"{MATERIALIZED_BUDGET / 2**30:.0f} GiB budget"}
    mws = torch.empty(need, dtype=torch.uint8, device=q.device)
    for _ in range(max(2, args.warmup)):
        R.relation_bwd_materialized(q, k, v, do, lam_t, workspace=mws)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    mk = max(5, K // 2)
    e0.record()
    for _ in range(mk):
        R.relation_bwd_materialized(q, k, v, do, lam_t, workspace=mws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / mk
    del mws
    return {"bwd_status": "ok", "bwd_ms": ms, "speedup_bwd": ms / bwd_ms,
            "step_ms": mat_fwd_ms + ms, "speedup_step": (mat_fwd_ms + ms) / (fwd_ms + bwd_ms)}


def layer_leg(hip, lib, K: int, warmup: int) -> dict:
    """The layer entry points at the paper's 100M geometry (4 x 8 heads of width
    80, T = 4096, RoPE base 1e4, Givens pairing A): whole-step time, the fused
    kernels' share (HIP events on their launch stream), and the rest, the
    layer's own linear passes, against the HBM peak."""
    import numpy as np
    import torch
    from paper_2608_20172_amd import binding as R
    from paper_2608_20172_amd.inputs import LAYER_WORKLOADS, make_givens_angles

    w = LAYER_WORKLOADS["paper100m_layer"]
    inp = make_workload_inputs(w)
    dev = torch.device("cuda:0")
    q, k, v, do = (torch.from_numpy(inp[n]).to(torch.bfloat16).to(dev) for n in ("q", "k", "v", "dout"))
    lam_t = torch.tensor([float(inp["lam"])], dtype=torch.float32, device=dev)
    th = torch.from_numpy(np.asarray(make_givens_angles(w.H), dtype=np.float32)).to(dev)
    kw = dict(pairing="A", rope_base=1.0e4)
    bws = torch.empty(max(1, R.relation_layer_bwd_workspace_bytes(q, **kw)), dtype=torch.uint8, device=dev)

    def step():
        f = R.relation_layer_fwd(q, k, v, lam_t, th, **kw)  # keeps the prepared operands for the backward
        g = R.relation_layer_bwd(q, k, v, f["o"], do, lam_t, f["row_stat"], th, saved=f["saved"], workspace=bws,
                                 **kw)
        return f, g

    for _ in range(max(2, warmup)):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(K):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / K

    def kernel_ms(name):
        ev = hip.events(2 * K)
        keep = arm(lib, name, ev)
        for _ in range(K):
            step()
        torch.cuda.synchronize()
        n = lib.relation_profile_disarm()
        del keep
        t = sum(hip.elapsed_ms(ev[2 * i], ev[2 * i + 1]) for i in range(n)) / max(n, 1)
        hip.destroy(ev)
        return t

    fused = kernel_ms("fwd") + kernel_ms("bwd")
    N, T, D, es = w.N, w.T, w.D, 2
    DP = 32 if D <= 32 else 64 if D <= 64 else 96 if D <= 96 else 128  # tiled width (bf16)
    row, prow = N * T * D * es, N * T * DP * es
    # algorithmic bytes of the layer's own passes in one step (the backward
    # reads the forward's prepared operands, so it prepares nothing again)
    fwd_bytes = 3 * row + 3 * prow + prow + row   # q, k, v in; rotated q, k, mixed v out; padded y to the caller
    bwd_bytes = (row + prow                       # dO padded
                 + 3 * prow + row + 3 * row)      # epilogue: padded gradients and v in, dq, dk, dv out
    passes_ms = ms - fused
    nbytes = fwd_bytes + bwd_bytes
    return {"workload": w.name, "B": w.B, "H": w.H, "T": w.T, "D": w.D, "padded_D": DP,
            "rope_base": 1.0e4, "givens": "A", "ms_per_step": ms, "tokens_per_s": w.tokens / (ms * 1e-3),
            "fused_kernels_ms": fused, "layer_passes_ms": passes_ms, "layer_passes_bytes": nbytes,
            "layer_passes_GBps": nbytes / (passes_ms * 1e-3) / 1e9 if passes_ms > 0 else None,
            "layer_passes_hbm_frac": nbytes / (passes_ms * 1e-3) / PEAK_HBM if passes_ms > 0 else None}


DECODE_SHAPES = [  # (name, B, H, cache length, D): one new token per sequence
    ("dec100m_T2048", 8, 12, 2048, 64),
    ("batch64_T4096", 64, 12, 4096, 64),
    ("long_T16384", 1, 16, 16384, 128),
]


def decode_leg(K: int) -> list:
    """relation_decode with full caches of bf16 Gaussians at three shapes:
    time per step and the algorithmic bytes (history K and V read once, the
    new token's q, k, v read, y written) against the HBM peak."""
    import numpy as np
    import torch
    from paper_2608_20172_amd import binding as R

    out = []
    rng = np.random.default_rng(11)
    for name, B, H, L, D in DECODE_SHAPES:
        dev = torch.device("cuda:0")
        std = 1.0 / math.sqrt(D)
        kc = (torch.randn(B, H, L, D, device=dev) * std).to(torch.bfloat16)
        vc = torch.randn(B, H, L, D, device=dev).to(torch.bfloat16)
        q = (torch.randn(B, H, D, device=dev) * std).to(torch.bfloat16)
        lens = torch.full((B,), L, dtype=torch.int32, device=dev)
        lam = torch.tensor([float(rng.normal(0, 0.02))], dtype=torch.float32, device=dev)
        ws = torch.empty(max(1, int(R.load_library().relation_decode_workspace_bytes(
            ctypes.byref(R.make_problem(kc))))), dtype=torch.uint8, device=dev)
        for _ in range(3):
            R.relation_decode(q, kc, vc, lens, lam, workspace=ws)
        torch.cuda.synchronize()
        n = max(10, K)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            R.relation_decode(q, kc, vc, lens, lam, workspace=ws)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / n
        nbytes = B * H * ((L - 1) * 2 * D * 2 + 4 * D * 2)
        out.append({"shape": name, "B": B, "H": H, "T": L, "D": D, "us_per_step": ms * 1e3,
                    "bytes": nbytes, "GBps": nbytes / (ms * 1e-3) / 1e9,
                    "hbm_frac": nbytes / (ms * 1e-3) / PEAK_HBM})
        del kc, vc, q, ws
    return out


LINEAR_SHAPES = [  # (B, H, T, D): one Linear Relation layer of 8 heads, width 64 (the paper's 48 and 60,
    (1, 8, 4096, 64),  # padded) and 128 (the paper's 80, padded)
    (1, 8, 16384, 64),
    (1, 8, 32768, 64),
    (1, 8, 4096, 128),
    (1, 8, 32768, 128),
]


def linear_leg(K: int) -> list:
    """relation_linear_fwd + relation_linear_bwd on bf16 Gaussians and
    log-retention -U(0, 0.05): time per step, tokens/s, the forward alone, and
    the step with the retention gate formed in the kernels and RoPE on p1, p2
    (the gated entry points, pre-activation r ~ N(0, 1))."""
    import torch
    from paper_2608_20172_amd import binding as R

    out = []
    for B, H, T, D in LINEAR_SHAPES:
        dev = torch.device("cuda:0")
        gen = torch.Generator(device=dev).manual_seed(5)
        p1, p2, v, dy = (torch.randn(B, H, T, D, device=dev, generator=gen).to(torch.bfloat16) for _ in range(4))
        g = -torch.rand(B, H, T, D, device=dev, generator=gen) * 0.05
        fws = torch.empty(max(1, int(R.load_library().relation_linear_fwd_workspace_bytes(
            ctypes.byref(R.make_problem(p1))))), dtype=torch.uint8, device=dev)
        bws = torch.empty(max(1, int(R.load_library().relation_linear_bwd_workspace_bytes(
            ctypes.byref(R.make_problem(p1))))), dtype=torch.uint8, device=dev)

        def fwd():
            return R.relation_linear_fwd(p1, p2, v, g, workspace=fws)

        def step():
            fwd()
            R.relation_linear_bwd(p1, p2, v, g, dy, workspace=bws)

        # the same step as the paper's layer runs it: the retention gate of eq. 15
        # formed in the kernels and RoPE on p1, p2 (over the paper's width 80
        # when the heads are 80 padded to 128)
        rope_dim = 80 if D == 128 else D
        r = torch.randn(B, H, T, D, device=dev, generator=gen)
        a_log = torch.full((H, D), -4.0, device=dev)   # -exp(-4) softplus(r - 3): alpha of about 0.999
        dt_bias = torch.full((H, D), -3.0, device=dev)
        gws = torch.empty(max(1, int(R.load_library().relation_linear_gated_bwd_workspace_bytes(
            ctypes.byref(R.make_problem(p1)), rope_dim))), dtype=torch.uint8, device=dev)
        gfws = torch.empty(max(1, int(R.load_library().relation_linear_gated_fwd_workspace_bytes(
            ctypes.byref(R.make_problem(p1)), rope_dim))), dtype=torch.uint8, device=dev)

        def gated_step():
            R.relation_linear_gated_fwd(p1, p2, v, r, a_log, dt_bias, rope_dim=rope_dim, workspace=gfws)
            R.relation_linear_gated_bwd(p1, p2, v, r, a_log, dt_bias, dy, rope_dim=rope_dim, workspace=gws)

        for _ in range(3):
            step()
        torch.cuda.synchronize()
        n = max(5, K // 3)
        res = {}
        for _ in range(3):
            gated_step()
        for name, fn in (("fwd_bwd", step), ("fwd", fwd), ("gated_fwd_bwd", gated_step)):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(n):
                fn()
            e1.record()
            torch.cuda.synchronize()
            res[name] = e0.elapsed_time(e1) / n
        out.append({"B": B, "H": H, "T": T, "D": D, "ms_fwd_bwd": res["fwd_bwd"], "ms_fwd": res["fwd"],
                    "tokens_per_s": B * T / (res["fwd_bwd"] * 1e-3), "ms_gated_fwd_bwd": res["gated_fwd_bwd"]})
        del p1, p2, v, dy, g, fws, bws, r, a_log, dt_bias, gws, gfws
    return out


def mfma_peak_leg(lib, hip) -> dict:
    """Achievable dense bf16 MFMA rate (relation_mfma_peak_probe: every SIMD
    runs independent 32x32x16 chains) and the shader clock during it, from the
    s_memtime / s_memrealtime differences of one wave (s_memrealtime runs at
    100 MHz), cross-checked against the event time."""
    import statistics
    import torch
    wg, iters = 256, 20000
    sink = torch.empty(wg * 256, dtype=torch.float32, device="cuda")
    clocks = torch.zeros(2, dtype=torch.int64, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    flops = float(lib.relation_mfma_peak_flops(wg, iters))
    ms, mhz = [], []
    for rep in range(6):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        if lib.relation_mfma_peak_probe(wg, iters, sink.data_ptr(), clocks.data_ptr(), stream) != 0:
            raise RuntimeError(lib.relation_last_error().decode())
        e1.record()
        torch.cuda.synchronize()
        if rep == 0:
            continue  # first launch loads the code object
        ms.append(e0.elapsed_time(e1))
        t, r = (int(x) for x in clocks.cpu().tolist())
        mhz.append(100.0 * t / r if r else float("nan"))
    med = statistics.median(ms)
    return {"tflops": flops / (med * 1e-3) / 1e12, "ms": med, "flops": flops,
            "clock_mhz_memtime": statistics.median(mhz),
            "note": "256 workgroups x 4 waves, 8 independent v_mfma_f32_32x32x16_bf16 chains per wave"}


def time_steps(fwd_call, bwd_call, K: int, warmup: int) -> dict:
    """Per-step event pairs around the forward and the backward call: means and
    medians of forward, backward and whole-step times (ms)."""
    import statistics
    import torch
    for _ in range(warmup):
        f = fwd_call()
        if bwd_call:
            bwd_call(f)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3 * K)]
    for s_ in range(K):
        ev[3 * s_].record()
        f = fwd_call()
        ev[3 * s_ + 1].record()
        if bwd_call:
            bwd_call(f)
        ev[3 * s_ + 2].record()
    torch.cuda.synchronize()
    fw = [ev[3 * i].elapsed_time(ev[3 * i + 1]) for i in range(K)]
    bw = [ev[3 * i + 1].elapsed_time(ev[3 * i + 2]) for i in range(K)] if bwd_call else [0.0] * K
    st = [a + b for a, b in zip(fw, bw)]
    return {"fwd_ms_mean": sum(fw) / K, "fwd_ms_median": statistics.median(fw),
            "bwd_ms_mean": sum(bw) / K, "bwd_ms_median": statistics.median(bw),
            "step_ms_mean": sum(st) / K, "step_ms_median": statistics.median(st)}


def workload_leg(name: str, K: int, warmup: int, peak_measured: float) -> dict:
    """One of the other decoder-scale workloads: forward (+ backward) tokens/s,
    TFLOP/s and fraction of the bf16 peaks (medians of per-step events), and
    the materialised baseline where its T x T workspace fits the budget."""
    import torch
    from paper_2608_20172_amd import binding as R
    w = WORKLOADS[name]
    inp = make_workload_inputs(w)
    dev = torch.device("cuda:0")
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    q, k, v = (torch.from_numpy(inp[n]).to(tdt).to(dev) for n in ("q", "k", "v"))
    do = torch.from_numpy(inp["dout"]).to(tdt).to(dev) if w.backward else None
    lam_t = torch.tensor([float(inp["lam"])], dtype=torch.float32, device=dev)
    ws = torch.empty(max(1, R.relation_bwd_workspace_bytes(q)), dtype=torch.uint8, device=dev)
    fwd_call = lambda: R.relation_fwd(q, k, v, lam_t)
    bwd_call = (lambda f: R.relation_bwd(q, k, v, f["o"], do, lam_t, f["row_stat"], workspace=ws)) \
        if w.backward else None
    n = max(10, K)
    t = time_steps(fwd_call, bwd_call, n, warmup)
    fl_f = flops(w, "fwd")
    fl_b = flops(w, "bwd") if w.backward else 0.0
    step = t["step_ms_median"]
    out = {"workload": w.name, "B": w.B, "H": w.H, "T": w.T, "D": w.D, "dtype": w.dtype,
           "passes": "fwd+bwd" if w.backward else "fwd", "steps": n, **t,
           "tokens_per_s": w.tokens / (step * 1e-3), "tflops": (fl_f + fl_b) / (step * 1e-3) / 1e12,
           "mfma_peak_frac": (fl_f + fl_b) / (step * 1e-3) / PEAK_BF16,
           "mfma_measured_peak_frac": (fl_f + fl_b) / (step * 1e-3) / (peak_measured * 1e12)
           if peak_measured else None,
           "fwd_tflops": fl_f / (t["fwd_ms_median"] * 1e-3) / 1e12}
    if w.backward:
        out["bwd_tflops"] = fl_b / (t["bwd_ms_median"] * 1e-3) / 1e12
    need = R.relation_fwd_materialized_workspace_bytes(q)
    if need > MATERIALIZED_BUDGET:
        out["materialized"] = {"status": f"skipped: T x T workspace {need / 2**30:.1f} GiB exceeds the "
                                         f"{MATERIALIZED_BUDGET / 2**30:.0f} GiB budget"}
    else:
        mws = torch.empty(need, dtype=torch.uint8, device=dev)
        mf = lambda: R.relation_fwd_materialized(q, k, v, lam_t, workspace=mws)
        mat = {"status": "ok"}
        mt = time_steps(mf, None, n, warmup)
        NTT = w.N * w.T * w.T
        es = 2 if w.dtype == "bf16" else 4
        mat["fwd_ms"] = mt["fwd_ms_median"]
        mat["speedup_fwd"] = mt["fwd_ms_median"] / t["fwd_ms_median"]
        mat["txt_hbm_GBps"] = NTT * (4 + 4 + es + es) / (mt["fwd_ms_median"] * 1e-3) / 1e9
        del mws
        if w.backward:
            nb = R.relation_bwd_materialized_workspace_bytes(q)
            if nb > MATERIALIZED_BUDGET:
                mat["bwd_status"] = "skipped: exceeds budget"
            else:
                bws = torch.empty(nb, dtype=torch.uint8, device=dev)
                mb = lambda: R.relation_bwd_materialized(q, k, v, do, lam_t, workspace=bws)
                bt = time_steps(mb, None, n, warmup)
                mat["bwd_ms"] = bt["fwd_ms_median"]
                mat["speedup_bwd"] = bt["fwd_ms_median"] / t["bwd_ms_median"]
                mat["speedup_step"] = (mat["fwd_ms"] + mat["bwd_ms"]) / step
                mat["bwd_txt_hbm_GBps"] = NTT * (8 + 8 + 2 * es + 2 * es) / (bt["fwd_ms_median"] * 1e-3) / 1e9
                del bws
        out["materialized"] = mat
    del q, k, v, do, ws
    torch.cuda.empty_cache()
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="dec100m_T2048", choices=sorted(WORKLOADS))
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-materialized", action="store_true")
    ap.add_argument("--no-layer", action="store_true", help="skip the layer entry points leg")
    ap.add_argument("--no-decode", action="store_true", help="skip the decode leg")
    ap.add_argument("--no-linear", action="store_true", help="skip the Linear Relation leg")
    ap.add_argument("--no-workloads", action="store_true", help="skip the other decoder-scale workloads")
    ap.add_argument("--copy-bytes", type=int, default=0)
    ap.add_argument("--copy-kind", choices=("memcpy", "elementwise"), default="elementwise")
    ap.add_argument("--summarize-counters", nargs=4, metavar=("FETCH", "WRITE", "COPY_FETCH", "COPY_WRITE"),
                    help="write the backward traffic file from four rocprofv3 --pmc CSVs "
                         "(needs --copy-bytes of the calibration copy)")
    args = ap.parse_args()

    if args.summarize_counters:
        t = summarize_counters(args.summarize_counters, args.copy_bytes)
        with open(TRAFFIC_FILE, "w") as f:
            json.dump(t, f, indent=1)
        print(json.dumps(t))
        return 0

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the fused operator is measured on one "
              "MI355X; multi-GPU runs are not part of this build.", file=sys.stderr)
        return 2
    if args.copy_bytes:
        copy_mode(args.copy_bytes, max(1, args.steps), args.copy_kind)
        return 0

    w = WORKLOADS[args.workload]
    inp = make_workload_inputs(w)
    lam = float(inp["lam"])

    # CPU baseline first, before anything initialises the GPU
    cpu = None
    if not args.no_cpu_baseline and w.backward:
        rounded = round_inputs(inp, w.dtype)
        lam32 = float(__import__("numpy").float32(lam))
        cpu = cpu_baseline(w, rounded, lam32, args.cpu_seconds)

    import torch
    from paper_2608_20172_amd import binding as R

    lib = R.load_library()
    hip = Hip()
    dev = torch.device("cuda:0")
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    q, k, v = (torch.from_numpy(inp[n]).to(tdt).to(dev) for n in ("q", "k", "v"))
    do = torch.from_numpy(inp["dout"]).to(tdt).to(dev) if w.backward else None
    lam_t = torch.tensor([lam], dtype=torch.float32, device=dev)
    ws = torch.empty(max(1, R.relation_bwd_workspace_bytes(q)), dtype=torch.uint8, device=dev)

    def step():
        f = R.relation_fwd(q, k, v, lam_t)
        if w.backward:
            R.relation_bwd(q, k, v, f["o"], do, lam_t, f["row_stat"], workspace=ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    K = args.steps
    # timed region: K whole steps; the library records HIP events on the launch
    # stream around the dominant kernel of every step: the fused dK/dV/dQ kernel
    # on the one-kernel backward (it does every product of the backward; the row
    # pass before it and the dq pass after it are O(T D) passes), the whole
    # two-kernel backward otherwise, the forward kernel for a forward-only workload
    fused = w.backward and w.dtype == "bf16" and w.D in (32, 64) and w.T >= 1536  # relation_bwd's one-kernel path
    main_kernel = ("bwd_dkdv" if fused else "bwd") if w.backward else "fwd"
    kev = hip.events(2 * K)
    keep = arm(lib, main_kernel, kev)
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for _ in range(K):
        step()
    t1.record()
    torch.cuda.synchronize()
    recorded = lib.relation_profile_disarm()
    del keep
    ms_step = t0.elapsed_time(t1) / K
    kern_ms = sum(hip.elapsed_ms(kev[2 * s], kev[2 * s + 1]) for s in range(recorded)) / max(recorded, 1)
    hip.destroy(kev)

    # forward / backward split of a step, means and medians of per-step events
    # (a separate pass: the extra events between the calls are kept out of the
    # timed region)
    split = time_steps(lambda: R.relation_fwd(q, k, v, lam_t),
                       (lambda f: R.relation_bwd(q, k, v, f["o"], do, lam_t, f["row_stat"], workspace=ws))
                       if w.backward else None, K, 0)
    fwd_ms, bwd_ms = split["fwd_ms_mean"], split["bwd_ms_mean"]

    # each fused kernel alone (further passes with the same launches)
    def kernel_ms(name, call):
        ev = hip.events(2 * K)
        kp = arm(lib, name, ev)
        for _ in range(K):
            call()
        torch.cuda.synchronize()
        nrec = lib.relation_profile_disarm()
        del kp
        ms = sum(hip.elapsed_ms(ev[2 * s], ev[2 * s + 1]) for s in range(nrec)) / max(nrec, 1)
        hip.destroy(ev)
        return ms

    fwd_kern_ms = kernel_ms("fwd", lambda: R.relation_fwd(q, k, v, lam_t))
    per_kernel = {"fwd_kernel_ms": fwd_kern_ms}
    if w.backward:
        f_saved = R.relation_fwd(q, k, v, lam_t)
        bcall = lambda: R.relation_bwd(q, k, v, f_saved["o"], do, lam_t, f_saved["row_stat"], workspace=ws)
        dcall = lambda: R.relation_bwd(q, k, v, f_saved["o"], do, lam_t, f_saved["row_stat"], workspace=ws,
                                       deterministic=True)
        per_kernel["bwd_path"] = "one kernel (dq by atomics)" if fused else "two kernels"
        per_kernel["bwd_dkdv_kernel_ms"] = kernel_ms("bwd_dkdv", bcall)
        if fused:
            per_kernel["bwd_prep_kernel_ms"] = kernel_ms("bwd_prep", bcall)
            per_kernel["bwd_convert_kernel_ms"] = kernel_ms("bwd_convert", bcall)
            per_kernel["bwd_deterministic_ms"] = kernel_ms("bwd", dcall)
            per_kernel["bwd_deterministic_dq_kernel_ms"] = kernel_ms("bwd_dq", dcall)
            per_kernel["bwd_deterministic_dkdv_kernel_ms"] = kernel_ms("bwd_dkdv", dcall)
        else:
            per_kernel["bwd_dq_kernel_ms"] = kernel_ms("bwd_dq", bcall)

    # materialised baseline forward
    mat = {"status": "skipped"}
    if not args.no_materialized:
        need = R.relation_fwd_materialized_workspace_bytes(q)
        if need > MATERIALIZED_BUDGET:
            mat = {"status": f"skipped: T x T workspace {need / 2**30:.1f} GiB exceeds the "
                              f"{MATERIALIZED_BUDGET / 2**30:.0f} GiB budget"}
        else:
            mws = torch.empty(need, dtype=torch.uint8, device=dev)
            for _ in range(max(2, args.warmup)):
                R.relation_fwd_materialized(q, k, v, lam_t, workspace=mws)
            torch.cuda.synchronize()
            m0 = torch.cuda.Event(enable_timing=True)
            m1 = torch.cuda.Event(enable_timing=True)
            mk = max(5, K // 2)
            m0.record()
            for _ in range(mk):
                R.relation_fwd_materialized(q, k, v, lam_t, workspace=mws)
            m1.record()
            torch.cuda.synchronize()
            mat_ms = m0.elapsed_time(m1) / mk
            NTT = w.N * w.T * w.T
            tt_bytes = NTT * (4 + 4 + 2 + 2)  # U written + read (fp32), F written + read (bf16)
            mat = {"status": "ok", "fwd_ms": mat_ms, "speedup_fwd": mat_ms / fwd_ms,
                   "txt_hbm_GBps": tt_bytes / (mat_ms * 1e-3) / 1e9}
            del mws
            if w.backward:
                mat.update(materialized_backward(w, q, k, v, do, lam_t, fwd_ms, bwd_ms, mat_ms, K, args))

    peak = mfma_peak_leg(lib, hip)
    legs = {"status": "skipped"}
    if not args.no_workloads:
        legs = {n: workload_leg(n, K, args.warmup, peak["tflops"])
                for n in ("dec10m_T512", "dec30m_T1024", "long_T16384") if n != w.name}
    layer = {"status": "skipped"}
    if not args.no_layer:
        layer = layer_leg(hip, lib, K, args.warmup)
    decode = {"status": "skipped"}
    if not args.no_decode:
        decode = decode_leg(K)
    linear = {"status": "skipped"}
    if not args.no_linear:
        linear = linear_leg(K)

    fl_f, fl_b = flops(w, "fwd"), flops(w, "bwd") if w.backward else 0.0
    kern_flops = fl_b if w.backward else fl_f
    achieved = kern_flops / (kern_ms * 1e-3)
    khash = sources_hash()
    traffic = traffic_for(khash, "bwd_fused_kernel" if fused else None) if w.backward else None
    out = {
        "metric": METRIC,
        "value": w.tokens / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "T": w.T, "D": w.D,
                   "passes": "fwd+bwd" if w.backward else "fwd", "boost_frac": w.boost_frac,
                   "parallelism": "single GPU"},
        "step_tflops": (fl_f + fl_b) / (ms_step * 1e-3) / 1e12,
        "mfma_peak_frac": (fl_f + fl_b) / (ms_step * 1e-3) / PEAK_BF16,
        "fwd_ms": fwd_ms,
        "bwd_ms": bwd_ms,
        "step_split_ms": split,
        "mfma_measured_peak": peak,
        "mfma_measured_peak_frac": (fl_f + fl_b) / (ms_step * 1e-3) / (peak["tflops"] * 1e12),
        "mfma_peak_frac_median_step": (fl_f + fl_b) / (split["step_ms_median"] * 1e-3) / PEAK_BF16,
        **per_kernel,
        "fwd_kernel_tflops": fl_f / (fwd_kern_ms * 1e-3) / 1e12,
        "materialized": mat,
        "layer": layer,
        "decode": decode,
        "linear": linear,
        "workloads": legs,
        "roofline": {
            "kernel": (("bwd_dkdv_kernel<PolBF16<%d>, %d, 8, true> (one-kernel backward: dK, dV and dQ)" % (w.D, w.D))
                       if fused else "relation_bwd (two kernels)") if w.backward else "fwd_kernel",
            "bound": "mfma",
            "achieved": achieved / 1e12,
            "peak": PEAK_BF16 / 1e12,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16,
            "traffic": traffic,
            "launches_timed": int(recorded),
            "kernel_ms": kern_ms,
            "sources_hash": khash,
            # the whole relation_bwd call (with the row pass and the dq pass) over the same flops
            "relation_bwd_ms": split["bwd_ms_median"] if w.backward else None,
            "relation_bwd_frac": (kern_flops / (split["bwd_ms_median"] * 1e-3) / PEAK_BF16) if w.backward else None,
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
