"""GPU parity of the attention-weight distillation loss (flex_awd_loss)
through the C ABI: the loss of every (b,h) slice and the gradients dW1, dW2,
dtau of their sum against the float64 oracle, on the same seeded inputs.

Tolerances: the fp32 path keeps every operand in fp32 (1e-4 relative); the
bf16 path rounds the features phi to bf16 before the A = phi phi^T products,
a relative perturbation of at most 2^-9 per feature, so A_ij moves by about
2^-9 of sum_f |phi_if psi_jf| (within 1.5 |A_ij| on these inputs) and log A,
the loss and dW by well under the 2e-2 bound used.  dtau = -sum_j g_j
||k_j||^2 / c over the keys is a sum of terms of both signs about twenty times
larger than the sum itself on these inputs, so its error is measured against
that absolute scale sum_j |g_j| ||k_j||^2 / c (simulating the bf16 feature
rounding in float64 gives 2e-3 of it at N = 2, 1e-4 at N >= 100)."""
import numpy as np
import pytest

import oracle as orc
import workloads as W
from tests.gpu_util import to_device, to_f64

pytestmark = pytest.mark.gpu

# (io, d, m, variant, B, H, N): ragged tails, a whole tile, the degenerate
# N = 1 (loss 0, gradient 0) and N = 2
CASES = [
    ("bf16", 64, 64, "nonstationary", 2, 2, 200),
    ("bf16", 64, 128, "stationary", 1, 3, 130),
    ("bf16", 64, 128, "nonstationary", 1, 2, 100),
    ("bf16", 32, 64, "nonstationary", 2, 1, 64),
    ("f32", 32, 64, "stationary", 1, 2, 77),
    ("f32", 32, 64, "nonstationary", 2, 2, 150),
    ("bf16", 64, 64, "nonstationary", 1, 2, 1),
    ("bf16", 64, 64, "stationary", 1, 1, 2),
]


@pytest.fixture(scope="module")
def F():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_27748_amd as F
    F.load()
    return F


def _rel(got, ref):
    n = np.linalg.norm(ref)
    return np.linalg.norm(got - ref) / n if n > 0 else np.linalg.norm(got)


def _dtau_scale(x, ref, variant):
    """sum over keys of |<phi(K_j), dphi(K_j)>| ||K_j||^2 / c, per head."""
    K = x.f64("K")
    pk = orc.feature_map(K, x.W1, x.W2, x.tau, variant)
    gk = (pk * ref["dphi_k"]).sum(-1)
    c = np.exp(x.tau.astype(np.float64))[None, :, None]
    return (np.abs(gk) * (K * K).sum(-1) / c).sum(axis=(0, 2))


def _check(io, out, ref, variant, x):
    tol = 2e-2 if io == "bf16" else 1e-4
    L, Lr = to_f64(out["loss"]), ref["loss"]
    assert np.all(np.isfinite(Lr))
    err = np.abs(L - Lr) / np.maximum(np.abs(Lr), 1e-2)
    assert err.max() <= tol, (err.max(), L, Lr)
    names = ["dW1"] + (["dW2"] if variant == "nonstationary" else [])
    for name in names:
        e = _rel(to_f64(out[name]), ref[name])
        assert e <= tol, (name, e)
    dt = to_f64(out["dtau"])
    # the floor covers N = 1, where dtau and its scale vanish (A_ij and den_i
    # are then the same sum taken in two orders, and the GPU leaves rounding of
    # order 1e-8); every other case here has a scale above 1e-3
    scale = np.maximum(_dtau_scale(x, ref, variant), np.abs(ref["dtau"]))
    e = np.abs(dt - ref["dtau"]) / np.maximum(scale, 1e-5)
    assert e.max() <= tol, ("dtau", e, dt, ref["dtau"])


@pytest.mark.parametrize("io,d,m,variant,B,H,N", CASES)
def test_awd_parity(F, io, d, m, variant, B, H, N):
    import torch
    wl = W.Workload("awd", B, H, N, d, m, variant, False, io, True, 2100 + N)
    x = W.generate_awd(wl)
    t = to_device(x)
    desc = F.make_desc(B, H, N, d, m, variant, False, io)
    out = F.flex_awd_loss(desc, t["Q"], t["K"], t["W1"], t["W2"], t["tau"])
    torch.cuda.synchronize()
    ref = orc.awd_grads(x.f64("Q"), x.f64("K"), x.W1, x.W2, x.tau, variant)
    _check(io, out, ref, variant, x)
    if N == 1:   # one key: A / den = 1 exactly, so the loss and the gradient vanish
        assert np.abs(to_f64(out["loss"])).max() < 1e-5
        assert np.abs(to_f64(out["dW1"])).max() < 1e-5


def test_awd_loss_only_matches(F):
    """dW1 = NULL computes the same loss without the gradient passes."""
    import torch
    wl = W.Workload("awd", 2, 2, 90, 64, 64, "nonstationary", False, "bf16", True, 2201)
    x = W.generate_awd(wl)
    t = to_device(x)
    desc = F.make_desc(2, 2, 90, 64, 64, "nonstationary", False, "bf16")
    a = F.flex_awd_loss(desc, t["Q"], t["K"], t["W1"], t["W2"], t["tau"])
    b = F.flex_awd_loss(desc, t["Q"], t["K"], t["W1"], t["W2"], t["tau"], grads=False)
    torch.cuda.synchronize()
    assert torch.equal(a["loss"], b["loss"])
    assert b["dW1"] is None


def test_awd_deterministic(F):
    """Two calls give bitwise equal losses and gradients."""
    import torch
    wl = W.Workload("awd", 2, 2, 300, 64, 128, "nonstationary", False, "bf16", True, 2202)
    x = W.generate_awd(wl)
    t = to_device(x)
    desc = F.make_desc(2, 2, 300, 64, 128, "nonstationary", False, "bf16")
    a = F.flex_awd_loss(desc, t["Q"], t["K"], t["W1"], t["W2"], t["tau"])
    b = F.flex_awd_loss(desc, t["Q"], t["K"], t["W1"], t["W2"], t["tau"])
    torch.cuda.synchronize()
    for k in ("loss", "dW1", "dW2", "dtau"):
        assert torch.equal(a[k], b[k]), k


def test_awd_full_size(F):
    """The distillation workload at its full size (B=32, H=8, N=512, d=64,
    m=64, nonstationary, bf16), in the launch configuration the benchmark
    times: every slice's loss and the whole gradient against the oracle."""
    import torch
    wl = W.AWD_WORKLOADS[W.AWD_HEADLINE]
    x = W.generate_awd(wl)
    t = to_device(x)
    desc = F.make_desc(wl.B, wl.H, wl.N, wl.d, wl.m, wl.variant, False, wl.io)
    out = F.flex_awd_loss(desc, t["Q"], t["K"], t["W1"], t["W2"], t["tau"])
    torch.cuda.synchronize()
    ref = orc.awd_grads(x.f64("Q"), x.f64("K"), x.W1, x.W2, x.tau, wl.variant)
    _check(wl.io, out, ref, wl.variant, x)


def test_awd_nan_where_the_ratio_is_not_positive(F):
    """The log is evaluated as printed: frequencies at pi between a query and a
    key give a negative kernel weight, and the GPU reports NaN for that slice
    exactly where the oracle does."""
    import torch
    B, H, N, d, m = 1, 2, 8, 32, 64
    r = np.random.default_rng(7)
    Q = np.zeros((B, H, N, d), np.float32)
    K = (r.standard_normal((B, H, N, d)) * 0.1).astype(np.float32)
    K[0, 0, 3, 0] = np.pi          # head 0: one key at pi along the first axis
    W1 = np.zeros((H, m, d), np.float32)
    W1[0, :, 0] = 1.0              # head 0: every frequency along that axis
    W1[1] = (r.standard_normal((m, d)) * 0.05).astype(np.float32)
    tau = np.full((H,), 3.0, np.float32)
    ref = orc.awd_loss(Q.astype(np.float64), K.astype(np.float64), W1, None, tau, "stationary")
    assert np.isnan(ref[0, 0]) and np.isfinite(ref[0, 1])
    desc = F.make_desc(B, H, N, d, m, "stationary", False, "f32")
    dev = lambda a: torch.from_numpy(a).cuda()
    out = F.flex_awd_loss(desc, dev(Q), dev(K), dev(W1), None, dev(tau), grads=False)
    torch.cuda.synchronize()
    L = to_f64(out["loss"])
    assert np.isnan(L[0, 0]) and abs(L[0, 1] - ref[0, 1]) <= 1e-4 * abs(ref[0, 1])
