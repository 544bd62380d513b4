"""Seeded synthetic inputs for the causal Full Relation operator.

This module only draws random numbers and names workload shapes. It holds none
of the operator's arithmetic, so both the HIP path and the fp64 oracle can be
fed from it without sharing any computation.

Draw order for one workload (numpy PCG64, ``default_rng(seed)``):
  1. Q, K, V ~ N(0, 1) * qkv_std       (each [B, H, T, D], fp64)
  2. dO ~ N(0, 1)                       (only when ``with_dout``)
  3. lambda ~ N(0, lam_std^2)           (one scalar, shared by all heads)
  4. row mask ~ Bernoulli(boost_frac)   (only when ``boost_frac > 0``); the Q
     rows it selects are multiplied by ``boost``.

Q and K stand for the relation projections after RoPE, V for the information
state after Givens mixing: the operator consumes exactly those per-head tensors.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, asdict

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    T: int
    D: int
    dtype: str          # "f32" or "bf16": storage type of q, k, v, o, dO and gradients
    qkv_std: float      # standard deviation of the Q, K, V draws
    backward: bool      # whether the workload includes the backward pass
    boost_frac: float = 0.0
    boost: float = 8.0
    lam_std: float = 0.02

    @property
    def N(self) -> int:
        return self.B * self.H

    @property
    def tokens(self) -> int:
        return self.B * self.T

    def describe(self) -> dict:
        d = asdict(self)
        d["N"] = self.N
        return d


def _std(D: int) -> float:
    return 1.0 / math.sqrt(D)


# The five decoder-scale workloads: a tiny fp32 forward check, then layers of
# roughly 10M / 30M / 100M-parameter decoders, then one long-context layer.
WORKLOADS = {
    "tiny_fp32": Workload("tiny_fp32", 1, 2, 128, 32, "f32", 1.0, False),
    "dec10m_T512": Workload("dec10m_T512", 8, 4, 512, 64, "bf16", _std(64), False),
    "dec30m_T1024": Workload("dec30m_T1024", 8, 8, 1024, 64, "bf16", _std(64), True),
    "dec100m_T2048": Workload("dec100m_T2048", 8, 12, 2048, 64, "bf16", _std(64), True,
                              boost_frac=0.05, boost=8.0),
    "long_T16384": Workload("long_T16384", 1, 16, 16384, 128, "bf16", _std(128), True),
}

# Layers at the paper's own model geometries (8 heads of width 48, 64, 80 and
# 60; context 1024, 2048, 4096 and 2048; the micro-batch of each scale), run
# through the layer entry points with RoPE and Givens mixing.
LAYER_WORKLOADS = {
    "paper10m_layer": Workload("paper10m_layer", 32, 8, 1024, 48, "bf16", _std(48), True),
    "paper30m_layer": Workload("paper30m_layer", 16, 8, 2048, 64, "bf16", _std(64), True),
    "paper100m_layer": Workload("paper100m_layer", 4, 8, 4096, 80, "bf16", _std(80), True),
    "hybrid30m_layer": Workload("hybrid30m_layer", 16, 8, 2048, 60, "bf16", _std(60), True),
}


def make_inputs(B: int, H: int, T: int, D: int, *, seed: int = 42, qkv_std: float = 1.0,
                with_dout: bool = True, lam_std: float = 0.02, lam: float | None = None,
                boost_frac: float = 0.0, boost: float = 8.0) -> dict:
    """Draw one seeded input set as fp64 numpy arrays of shape [B, H, T, D].

    ``lam`` overrides the drawn lambda (the draw still happens so that the
    stream position of later draws does not depend on the override).
    """
    rng = np.random.default_rng(seed)
    shape = (B, H, T, D)
    q = rng.standard_normal(shape) * qkv_std
    k = rng.standard_normal(shape) * qkv_std
    v = rng.standard_normal(shape) * qkv_std
    dout = rng.standard_normal(shape) if with_dout else None
    lam_drawn = float(rng.normal(0.0, lam_std))
    if boost_frac > 0.0:
        mask = rng.random((B, H, T)) < boost_frac
        q[mask] *= boost
    else:
        mask = np.zeros((B, H, T), dtype=bool)
    return {
        "q": q, "k": k, "v": v, "dout": dout,
        "lam": lam_drawn if lam is None else float(lam),
        "boost_mask": mask,
    }


def make_givens_angles(H: int, seed: int = 42, spread: float = math.pi) -> np.ndarray:
    """H/2 head-pair angles ~ U(-spread, spread), fp64, from a stream of their
    own (the paper initialises them to zero; tests need general angles)."""
    rng = np.random.default_rng(seed + 7919)
    return rng.uniform(-spread, spread, H // 2)


def make_log_retention(B: int, H: int, T: int, D: int, seed: int = 42, gmax: float = 0.5) -> np.ndarray:
    """Per-channel log-retention values ~ -U(0, gmax), [B, H, T, D] fp64, from
    a stream of their own (retention alpha = exp(g) in (exp(-gmax), 1])."""
    rng = np.random.default_rng(seed + 104729)
    return -rng.uniform(0.0, gmax, (B, H, T, D))


def make_workload_inputs(w: Workload, seed: int = 42, lam: float | None = None) -> dict:
    return make_inputs(w.B, w.H, w.T, w.D, seed=seed, qkv_std=w.qkv_std,
                       with_dout=w.backward, lam_std=w.lam_std, lam=lam,
                       boost_frac=w.boost_frac, boost=w.boost)


def make_sharp_inputs(B: int, H: int, T: int, D: int, *, seed: int = 42,
                      with_dout: bool = True, lam: float | None = None) -> dict:
    """Inputs whose pairwise evidence reaches tens of units: Q, K ~ N(0, 1)
    without the 1/sqrt(D) factor and 5% of Q rows boosted x8, so the running
    maximum of the Exchange scan actually moves."""
    return make_inputs(B, H, T, D, seed=seed, qkv_std=1.0, with_dout=with_dout,
                       lam=lam, boost_frac=0.05, boost=8.0)
