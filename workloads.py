"""Seeded synthetic workloads for the RFF linear-attention hot path.

This module holds the workload shapes and the seeded input generator, and
nothing of the method's arithmetic: it only draws random numbers and rounds
them to the storage precision.  Both the float64 oracle and the GPU path
consume exactly the arrays produced here.

Recipe (stand-in for the paper's LRA / WikiText-103 workloads, which are not
available here): for workload seed ``s`` a ``numpy.random.default_rng(s)``
draws, in this order and each standard normal float64 in C order,
W1 [H,m,d], W2 [H,m,d] (nonstationary only), Q, K [B,H,N,d], V [B,H,N,dv]
and dO [B,H,N,dv] (workloads with a backward pass; dv = d unless a workload
sets it).  W is rounded to fp32
(round-to-nearest-even).  Q, K, V are multiplied by d^-1/4 and rounded to the
storage dtype (fp32, or bf16 via fp32 with round-to-nearest-even).  dO is
rounded the same way, without the scale.  tau = ln 2 for every head and
sigma = 1.

Frequencies are drawn independently per head, following the paper's
parameter analysis (Appendix B, per-head frequencies).  With inputs scaled
by d^-1/4 the softmax bandwidth 2*sqrt(d) of the norm factor (Sec. 3.1) is
exp(tau) = 2 in these units.
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
    N: int
    d: int
    m: int
    variant: str        # "stationary" | "nonstationary"
    causal: bool
    io: str             # "f32" | "bf16"
    backward: bool
    seed: int
    chunk: int = 64
    value_dim: int = 0  # d_v; 0 means d_v = d

    @property
    def dv(self) -> int:
        return self.value_dim or self.d

    @property
    def dprime(self) -> int:
        return 2 * self.m

    def scaled(self, **kw) -> "Workload":
        d = asdict(self)
        d.update(kw)
        return Workload(**d)


# The five configurations of the hot path plus the headline training shape
# (causal, nonstationary, fwd+bwd, N=8192, d=64, m=128 per frequency matrix).
WORKLOADS = {
    "tiny_stationary_noncausal_f32": Workload(
        "tiny_stationary_noncausal_f32", 1, 1, 256, 32, 64,
        "stationary", False, "f32", False, 1001),
    "lm_stationary_causal": Workload(
        "lm_stationary_causal", 8, 12, 1024, 64, 128,
        "stationary", True, "bf16", False, 1002),
    "nonstationary_causal_train": Workload(
        "nonstationary_causal_train", 4, 16, 4096, 64, 128,
        "nonstationary", True, "bf16", True, 1003),
    "long_stationary_noncausal": Workload(
        "long_stationary_noncausal", 16, 8, 16384, 64, 64,
        "stationary", False, "bf16", False, 1004),
    "train_at_scale_d128": Workload(
        "train_at_scale_d128", 2, 16, 8192, 128, 256,
        "nonstationary", True, "bf16", True, 1005),
    "headline_causal_train_d64": Workload(
        "headline_causal_train_d64", 2, 16, 8192, 64, 128,
        "nonstationary", True, "bf16", True, 1006),
}
HEADLINE = "headline_causal_train_d64"

# Attention-weight distillation (the loss of App. A.3, used in Sec. 4.3):
# non-causal, the softmax target from the same Q and K.  Stand-in for the
# paper's GLUE distillation of a RoBERTa-size encoder (8 heads of d = 64,
# batch 32, n = d frequencies, sequences up to 512 tokens); those data are not
# available here and are not needed: the loss and its gradient cost the same
# for any values.
AWD_WORKLOADS = {
    "distill_glue_B32_H8_N512_d64_m64": Workload(
        "distill_glue_B32_H8_N512_d64_m64", 32, 8, 512, 64, 64,
        "nonstationary", False, "bf16", True, 2001),
}
AWD_HEADLINE = "distill_glue_B32_H8_N512_d64_m64"


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round-to-nearest-even); uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = np.isnan(x)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    if nan.any():
        r = np.where(nan, np.uint16(0x7FC0), r)
    return r


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@dataclass
class Inputs:
    """Storage-precision inputs.  ``Q``/``K``/``V``/``dO`` are float32 arrays
    for the fp32 path or uint16 bfloat16 bit patterns for the bf16 path."""
    wl: Workload
    W1: np.ndarray
    W2: np.ndarray | None
    tau: np.ndarray
    Q: np.ndarray
    K: np.ndarray
    V: np.ndarray
    dO: np.ndarray | None
    sigma: float = 1.0

    def f64(self, name: str) -> np.ndarray | None:
        """The stored values of one input, widened exactly to float64."""
        a = getattr(self, name)
        if a is None:
            return None
        if a.dtype == np.uint16:
            return bf16_bits_to_f64(a)
        return a.astype(np.float64)


def _store(x: np.ndarray, io: str) -> np.ndarray:
    x32 = x.astype(np.float32)
    if io == "f32":
        return x32
    if io == "bf16":
        return f32_to_bf16_bits(x32)
    raise ValueError(io)


def generate(wl: Workload, seed: int | None = None, with_grad: bool | None = None) -> Inputs:
    """Draw the seeded inputs of a workload (see the module docstring)."""
    rng = np.random.default_rng(wl.seed if seed is None else seed)
    H, m, d = wl.H, wl.m, wl.d
    W1 = rng.standard_normal((H, m, d)).astype(np.float32)
    W2 = (rng.standard_normal((H, m, d)).astype(np.float32)
          if wl.variant == "nonstationary" else None)
    shp = (wl.B, wl.H, wl.N, wl.d)
    scale = d ** -0.25
    Q = _store(rng.standard_normal(shp) * scale, wl.io)
    K = _store(rng.standard_normal(shp) * scale, wl.io)
    V = _store(rng.standard_normal((wl.B, wl.H, wl.N, wl.dv)) * scale, wl.io)
    want_grad = wl.backward if with_grad is None else with_grad
    dO = _store(rng.standard_normal((wl.B, wl.H, wl.N, wl.dv)), wl.io) if want_grad else None
    tau = np.full((H,), math.log(2.0), dtype=np.float32)
    return Inputs(wl, W1, W2, tau, Q, K, V, dO)


def generate_awd(wl: Workload, seed: int | None = None) -> Inputs:
    """Seeded inputs of a distillation-loss workload.

    A ``numpy.random.default_rng(seed)`` draws, in this order and each standard
    normal float64 in C order, W1 [H,m,d], W2 [H,m,d] (nonstationary only), Q
    and K [B,H,N,d].  W is multiplied by 0.5 / sqrt(d) and rounded to fp32; Q
    and K keep unit-variance entries (logits Q.K / sqrt(d) of unit variance,
    as in a trained attention layer) and are rounded to the storage dtype;
    tau = ln(2d) for every head.  With these frequencies and this bandwidth the
    projections stay within about one radian, so every kernel weight
    phi(Q_i)^T phi(K_j) is positive and the loss's logarithm is defined: a
    kernel initialised near a wide Gaussian before distillation.  No V or dO.
    """
    rng = np.random.default_rng(wl.seed if seed is None else seed)
    H, m, d = wl.H, wl.m, wl.d
    ws = 0.5 / math.sqrt(d)
    W1 = (rng.standard_normal((H, m, d)) * ws).astype(np.float32)
    W2 = ((rng.standard_normal((H, m, d)) * ws).astype(np.float32)
          if wl.variant == "nonstationary" else None)
    shp = (wl.B, wl.H, wl.N, wl.d)
    Q = _store(rng.standard_normal(shp), wl.io)
    K = _store(rng.standard_normal(shp), wl.io)
    tau = np.full((H,), math.log(2.0 * d), dtype=np.float32)
    return Inputs(wl, W1, W2, tau, Q, K, None, None)
