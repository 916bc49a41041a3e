"""The bf16 rounding floor of the backward against the number of frequencies.

The float64 oracle backward is run twice on the inputs of the bf16 parity
tests: exactly, and with only the feature maps phi(Q), phi(K) rounded to bf16
(round to nearest even), as the GPU rounds them for its MFMA operands.  The
gap is a floor that the bf16 path cannot beat.  Few frequencies average the
rounding less: at m = 16 the floor alone reaches the 2e-2 bar of the bf16
gradient checks, at m = 128 it is a third of it.  This is why the bf16
gradient parity tests start at m = 48 (the fp32 path is tested at m = 16).
"""
import numpy as np
import pytest

import workloads as W
import oracle.flex_oracle as orc
from tests.parity import frob_rel, KAPPA_MAX


def _bf16(x):
    x = np.ascontiguousarray(np.asarray(x, np.float32))
    u = x.view(np.uint32)
    r = ((u >> 16) & 1) + 0x7FFF
    return ((u + r) & 0xFFFF0000).astype(np.uint32).view(np.float32).astype(np.float64)


def _floor(d, m, variant, monkeypatch, shape=(2, 2, 200), causal=False, seed=21):
    wl = W.Workload("small", *shape, d, m, variant, causal, "bf16", True, seed)
    x = W.generate(wl)
    kap = orc.conditioning(x.f64("Q"), x.f64("K"), x.W1, x.W2, x.tau, variant, causal)
    x.dO = x.dO * (kap <= KAPPA_MAX["bf16"])[..., None].astype(x.dO.dtype)
    args = (x.f64("Q"), x.f64("K"), x.f64("V"), x.W1, x.W2, x.tau, x.f64("dO"), variant, causal)
    ref = orc.linattn_bwd(*args)
    exact = orc.feature_map_parts
    with monkeypatch.context() as mp:
        mp.setattr(orc, "feature_map_parts", lambda *a, **k: (lambda r: (_bf16(r[0]), r[1]))(exact(*a, **k)))
        got = orc.linattn_bwd(*args)
    return max(frob_rel(got[k], ref[k]) for k in ("dQ", "dK", "dW1"))


def test_bf16_rounding_floor_against_m(monkeypatch):
    few = _floor(32, 16, "nonstationary", monkeypatch)
    many = _floor(64, 128, "nonstationary", monkeypatch)
    assert few > 1.5e-2          # at m = 16 the floor alone nears the 2e-2 bar
    assert many < 1e-2           # at m = 128 it is well under it
    assert few > 2.5 * many


def test_bf16_rounding_floor_m48_short_causal(monkeypatch):
    """A drawn input at m = 48 (B=1, H=2, N=65, d=64, causal): the feature
    rounding alone costs 1.7 % of dQ, so the bf16 path's other roundings can
    take it past the 2e-2 bar (the GPU gives 2.6 %).  The randomized parity
    test checks bf16 gradients from m = 64."""
    f = _floor(64, 48, "nonstationary", monkeypatch, shape=(1, 2, 65), causal=True, seed=1173)
    assert 1.5e-2 < f < 2e-2


def test_bf16_forward_rounding_floor_m16_short():
    """The bf16 causal forward rounds the features, the intra-chunk kernel
    matrix (for A [V | 1]) and the carried state (the readout's operand) to
    bf16.  Emulated in float64 on a drawn input with m = 16 and N = 17 (B=1,
    H=2, d = d_v = 128, 16-token chunks), those roundings alone put T2 past
    the 2e-2 bar (the GPU gives 2.1 %); the randomized test checks T2 for bf16
    from m = 48."""
    from tests.parity import KAPPA_MAX as KF
    wl = W.Workload("floor_fwd", 1, 2, 17, 128, 16, "nonstationary", True, "bf16", False, 1336, value_dim=128)
    x = W.generate(wl)
    Q, K, V = x.f64("Q"), x.f64("K"), x.f64("V")
    O, _ = orc.linattn_fwd(Q, K, V, x.W1, x.W2, x.tau, wl.variant, True)
    pq = _bf16(orc.feature_map(Q, x.W1, x.W2, x.tau, wl.variant))
    pk = _bf16(orc.feature_map(K, x.W1, x.W2, x.tau, wl.variant))
    Vp = np.concatenate([V, np.ones(V.shape[:-1] + (1,))], -1)
    out = np.zeros(Vp.shape)
    C = 16
    for h in range(wl.H):
        S = np.zeros((2 * wl.m, wl.dv + 1))
        for c0 in range(0, wl.N, C):
            c1 = min(wl.N, c0 + C)
            A = np.tril(pq[0, h, c0:c1] @ pk[0, h, c0:c1].T)
            out[0, h, c0:c1] = _bf16(A) @ Vp[0, h, c0:c1] + pq[0, h, c0:c1] @ _bf16(S)
            S = S + pk[0, h, c0:c1].T @ Vp[0, h, c0:c1]
    Oe = out[..., :-1] / out[..., -1:]
    kap = orc.conditioning(Q, K, x.W1, x.W2, x.tau, wl.variant, True)
    good = kap <= KF["bf16"]
    assert frob_rel(Oe[good], O[good]) > 2e-2
