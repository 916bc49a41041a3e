"""GPU parity of the backward pass (dQ, dK, dV, dW1, dW2, dtau) against the
float64 oracle, through the C ABI.

Criterion T3 (tests/parity.py): the upstream gradient is zeroed on rows whose
denominator is ill-conditioned (kappa_i > kappa_max), identically for the GPU
and the oracle; then every gradient's Frobenius relative error must be within
the tolerance.
"""
import numpy as np
import pytest

import oracle as orc
import workloads as W
from tests.gpu_util import to_device, to_f64, desc_of
from tests.parity import check_grads, check_grad_rows, dv_row_scale, dtau_scale, KAPPA_MAX_GRAD as KAPPA_MAX, TOL

pytestmark = pytest.mark.gpu

SHAPES = [("f32", 32, 64), ("bf16", 32, 64), ("bf16", 64, 64), ("bf16", 64, 128), ("bf16", 128, 256),
          # frequency groups at the other shapes, some with a padded first group
          # (bf16 from m = 48: below that, rounding the features to bf16 alone
          # puts the gradients at the 2e-2 bar)
          ("f32", 32, 128), ("bf16", 32, 192), ("bf16", 64, 256), ("bf16", 128, 64), ("bf16", 128, 128),
          ("f32", 32, 16), ("bf16", 64, 48), ("bf16", 128, 80), ("f32", 32, 96)]


@pytest.fixture(scope="module")
def F():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_27748_amd as F
    F.load()
    return F


def masked_inputs(wl, x):
    """Zero dO on rows with kappa > kappa_max (stored precision kept); returns
    the condition numbers."""
    kap = orc.conditioning(x.f64("Q"), x.f64("K"), x.W1, x.W2, x.tau, wl.variant, wl.causal)
    keep = kap <= KAPPA_MAX[wl.io]
    x.dO = x.dO * keep[..., None].astype(x.dO.dtype)
    return kap


def check_rows(wl, x, got, ref, kap):
    """Row-wise gradient checks (tests/parity.py check_grad_rows), for slices
    of at least 32 rows."""
    if wl.N < 32:
        return None
    pq = orc.feature_map(x.f64("Q"), x.W1, x.W2, x.tau, wl.variant)
    pk = orc.feature_map(x.f64("K"), x.W1, x.W2, x.tau, wl.variant)
    sc = dv_row_scale(pq, pk, x.f64("dO"), ref["den"], kap, wl.causal)
    return check_grad_rows(wl.io, got, ref, dv_scale=sc, n_terms=wl.N)


def gpu_fwd_bwd(F, wl, x, segments=0, reuse=False):
    """Forward then backward through the C ABI; with reuse=True the backward
    is given the forward's workspace (its segment states are reused)."""
    import torch
    t = to_device(x)
    d = desc_of(wl, segments=segments)
    ws_f = torch.empty(F.workspace_size(d, F.FLEX_PASS_FWD) + 256, dtype=torch.uint8, device=t["Q"].device)
    O, den = F.flex_linattn_fwd(d, t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"], ws=ws_f)
    g = F.flex_linattn_bwd(d, t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"], O, den, t["dO"],
                           fwd_ws=ws_f if reuse else None)
    return {k: (None if v is None else to_f64(v)) for k, v in g.items()}


def oracle_bwd(wl, x):
    """Oracle gradients and the dtau scale of T3."""
    ref = orc.linattn_bwd(x.f64("Q"), x.f64("K"), x.f64("V"), x.W1, x.W2, x.tau, x.f64("dO"),
                          wl.variant, wl.causal, return_aux=True)
    return ref, {"dtau": dtau_scale(x, wl, ref)}


def names_of(wl):
    return ["dQ", "dK", "dV", "dW1", "dtau"] + (["dW2"] if wl.variant == "nonstationary" else [])


@pytest.mark.parametrize("reuse", [False, True])
@pytest.mark.parametrize("io,d,m", SHAPES)
@pytest.mark.parametrize("variant", ["stationary", "nonstationary"])
@pytest.mark.parametrize("causal", [False, True])
def test_backward_small(F, io, d, m, variant, causal, reuse):
    wl = W.Workload("small", 2, 2, 200, d, m, variant, causal, io, True, 21)
    x = W.generate(wl)
    kap = masked_inputs(wl, x)
    got = gpu_fwd_bwd(F, wl, x, reuse=reuse)
    ref, sc = oracle_bwd(wl, x)
    check_grads(io, got, ref, names_of(wl), sc)
    check_rows(wl, x, got, ref, kap)


@pytest.mark.parametrize("d,dv", [(64, 32), (128, 64), (128, 32), (32, 64), (64, 128), (32, 128)])
@pytest.mark.parametrize("variant", ["stationary", "nonstationary"])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("reuse", [False, True])
def test_backward_value_width(F, d, dv, variant, causal, reuse):
    """d_v != d: the backward at width max(d, d_v) on zero-padded copies."""
    wl = W.Workload("dv", 2, 2, 150, d, 80, variant, causal, "bf16", True, 63, value_dim=dv)
    x = W.generate(wl)
    kap = masked_inputs(wl, x)
    got = gpu_fwd_bwd(F, wl, x, reuse=reuse)
    assert got["dQ"].shape == (2, 2, 150, d) and got["dV"].shape == (2, 2, 150, dv)
    assert got["dW1"].shape == (2, 80, d)
    ref, sc = oracle_bwd(wl, x)
    check_grads("bf16", got, ref, names_of(wl), sc)
    check_rows(wl, x, got, ref, kap)


@pytest.mark.parametrize("reuse", [False, True])
@pytest.mark.parametrize("segments", [1, 2, 3])
@pytest.mark.parametrize("causal", [False, True])
def test_backward_segments(F, segments, causal, reuse):
    wl = W.Workload("seg", 1, 2, 330, 64, 128, "nonstationary", causal, "bf16", True, 23)
    x = W.generate(wl)
    kap = masked_inputs(wl, x)
    got = gpu_fwd_bwd(F, wl, x, segments=segments, reuse=reuse)
    ref, sc = oracle_bwd(wl, x)
    check_grads("bf16", got, ref, names_of(wl), sc)
    check_rows(wl, x, got, ref, kap)


@pytest.mark.parametrize("segments", [1, 2])
@pytest.mark.parametrize("variant", ["stationary", "nonstationary"])
def test_backward_f32_long_sweep(F, segments, variant):
    """fp32, 2048 tokens in one or two sequential sweeps: the carried states
    take ~1000 MFMA k-steps each, rounded once per 32 tokens.  (With a
    rounding per 4-token MFMA, dQ reached 1.1e-4 here, over the 1e-4 bar.)"""
    wl = W.Workload("f32long", 1, 3, 2048, 32, 64, variant, True, "f32", True, 1062)
    x = W.generate(wl)
    kap = masked_inputs(wl, x)
    got = gpu_fwd_bwd(F, wl, x, segments=segments)
    ref, sc = oracle_bwd(wl, x)
    check_grads("f32", got, ref, names_of(wl), sc)
    check_rows(wl, x, got, ref, kap)


@pytest.mark.parametrize("reuse", [False, True])
def test_backward_many_segments(F, reuse):
    """12 segments: the carry-ins of both states come from the scans (up to a
    few segments the sweeps sum them from the local states themselves)."""
    wl = W.Workload("manyseg", 1, 2, 900, 64, 128, "nonstationary", True, "bf16", True, 37)
    x = W.generate(wl)
    kap = masked_inputs(wl, x)
    got = gpu_fwd_bwd(F, wl, x, segments=12, reuse=reuse)
    ref, sc = oracle_bwd(wl, x)
    check_grads("bf16", got, ref, names_of(wl), sc)
    check_rows(wl, x, got, ref, kap)


@pytest.mark.parametrize("reuse", [False, True])
def test_backward_128_segments(F, reuse):
    """128 segments of one 64-token chunk each (small B*H, long N takes up to
    one segment per CU): scans over 128 states, 128 frequency-gradient
    partials per head."""
    wl = W.Workload("seg128", 1, 1, 128 * 64 - 17, 32, 64, "nonstationary", True, "bf16", True, 41)
    x = W.generate(wl)
    kap = masked_inputs(wl, x)
    got = gpu_fwd_bwd(F, wl, x, segments=128, reuse=reuse)
    ref, sc = oracle_bwd(wl, x)
    check_grads("bf16", got, ref, names_of(wl), sc)
    check_rows(wl, x, got, ref, kap)


def test_backward_256_segments(F):
    """256 segments, the most the heuristic takes (N = 16379: 256 chunks, the
    last of 59 tokens), with the forward's states: scans over 256 states, R'
    suffixes from the scan, 256 frequency-gradient partials per head."""
    wl = W.Workload("seg256", 1, 1, 256 * 64 - 5, 32, 64, "nonstationary", True, "bf16", True, 43)
    x = W.generate(wl)
    kap = masked_inputs(wl, x)
    got = gpu_fwd_bwd(F, wl, x, segments=256, reuse=True)
    ref, sc = oracle_bwd(wl, x)
    check_grads("bf16", got, ref, names_of(wl), sc)
    check_rows(wl, x, got, ref, kap)


@pytest.mark.parametrize("reuse", [False, True])
def test_backward_many_partials(F, reuse):
    """B = 3 and 7 segments give 42 frequency-gradient partials per head: the
    reduce takes them in two batches, the second one partly past the list."""
    wl = W.Workload("partials", 3, 2, 500, 64, 64, "nonstationary", True, "bf16", True, 33)
    x = W.generate(wl)
    kap = masked_inputs(wl, x)
    got = gpu_fwd_bwd(F, wl, x, segments=7, reuse=reuse)
    ref, sc = oracle_bwd(wl, x)
    check_grads("bf16", got, ref, names_of(wl), sc)
    check_rows(wl, x, got, ref, kap)


@pytest.mark.parametrize("reuse", [False, True])
@pytest.mark.parametrize("N", [2, 64, 65, 1050])
def test_backward_edge_lengths(F, N, reuse):
    """Ragged lengths; 1050 with 3 segments leaves forward and backward chunk
    counts whose segment boundaries only agree when the backward follows the
    forward's segments."""
    wl = W.Workload("edge", 1, 2, N, 64, 64, "nonstationary", True, "bf16", True, 25)
    x = W.generate(wl)
    kap = masked_inputs(wl, x)
    got = gpu_fwd_bwd(F, wl, x, segments=3 if N > 1000 else 0, reuse=reuse)
    ref, sc = oracle_bwd(wl, x)
    check_grads("bf16", got, ref, names_of(wl), sc)
    check_rows(wl, x, got, ref, kap)


@pytest.mark.parametrize("d,m", [(64, 128), (128, 256)])
def test_backward_reuse_matches_recompute(F, d, m):
    """The backward with the forward's segment states and the backward that
    recomputes them differ only in the rounding of those states.  With the
    states passed in, the dQ sweep also forms the query-side R' locals that the
    pre-pass forms otherwise, from the same operands in the same order."""
    wl = W.Workload("reuse", 2, 2, 700 if d == 64 else 300, d, m, "nonstationary", True, "bf16", True, 31)
    x = W.generate(wl)
    masked_inputs(wl, x)
    a = gpu_fwd_bwd(F, wl, x, reuse=False)
    b = gpu_fwd_bwd(F, wl, x, reuse=True)
    for k in ("dK", "dV"):
        np.testing.assert_array_equal(a[k], b[k])   # key side: same R' path
    for k in ("dQ", "dW1", "dW2"):
        assert np.linalg.norm(a[k] - b[k]) <= 1e-3 * np.linalg.norm(a[k]), k


@pytest.mark.parametrize("causal", [False, True])
def test_backward_single_token(F, causal):
    """N = 1: O_0 = V_0 whatever the features, so dV = dO and every other
    gradient vanishes.  The GPU values must be zero up to rounding, measured
    against the size the same product chain has for a generic row:
    |dO| |V| |phi(Q)| |phi(K)| / |den| times |W| (and |k|^2/c for dtau)."""
    wl = W.Workload("one", 1, 2, 1, 64, 64, "nonstationary", causal, "bf16", True, 29)
    x = W.generate(wl)
    got = gpu_fwd_bwd(F, wl, x)
    dO, V, Q, K = x.f64("dO"), x.f64("V"), x.f64("Q"), x.f64("K")
    np.testing.assert_allclose(got["dV"], dO, rtol=2e-2, atol=1e-6)
    pq = orc.feature_map(Q, x.W1, x.W2, x.tau, wl.variant)
    pk = orc.feature_map(K, x.W1, x.W2, x.tau, wl.variant)
    den = np.abs((pq * pk).sum(-1))
    chain = (np.linalg.norm(dO, axis=-1) * np.linalg.norm(V, axis=-1)
             * np.linalg.norm(pq, axis=-1) * np.linalg.norm(pk, axis=-1) / den)[0, :, 0]
    wn = np.array([np.linalg.norm(x.W1[h]) + np.linalg.norm(x.W2[h]) for h in range(wl.H)])
    for n, scale in [("dQ", chain * wn), ("dK", chain * wn), ("dW1", chain * wn),
                     ("dW2", chain * wn), ("dtau", chain * (K * K).sum(-1)[0, :, 0] / 2.0)]:
        g = got[n]
        for h in range(wl.H):
            gh = g[:, h] if n in ("dQ", "dK") else g[h]
            assert np.linalg.norm(gh) <= TOL["bf16"] * scale[h], (n, h, np.linalg.norm(gh), scale[h])


def test_backward_deterministic(F):
    import torch
    wl = W.Workload("det", 2, 2, 300, 64, 128, "nonstationary", True, "bf16", True, 27)
    x = W.generate(wl)
    t = to_device(x)
    d = desc_of(wl)
    O, den = F.flex_linattn_fwd(d, t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"])
    g1 = F.flex_linattn_bwd(d, t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"], O, den, t["dO"])
    g2 = F.flex_linattn_bwd(d, t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"], O, den, t["dO"])
    torch.cuda.synchronize()
    for k in g1:
        if g1[k] is not None:
            assert torch.equal(g1[k], g2[k]), k


def _slice_bwd_oracle(wl, x, b, h):
    sl = (slice(b, b + 1), slice(h, h + 1))
    W2 = None if x.W2 is None else x.W2[h:h + 1]
    ref = orc.linattn_bwd(x.f64("Q")[sl], x.f64("K")[sl], x.f64("V")[sl], x.W1[h:h + 1], W2,
                          x.tau[h:h + 1], x.f64("dO")[sl], wl.variant, wl.causal, return_aux=True)
    K = x.f64("K")[sl]
    c = np.exp(np.float64(x.tau[h]))
    ref["tau_scale"] = float((np.abs(ref["phi_k"] * ref["dphi_k"]).sum(-1) * (K * K).sum(-1) / c).sum())
    return ref


@pytest.mark.parametrize("name", ["nonstationary_causal_train", "train_at_scale_d128", "headline_causal_train_d64"])
def test_backward_full_size_sampled(F, name):
    """Full configured size, default launch configuration.  For two heads (the
    first and the last), every slice's dQ, dK, dV rows and the head's dW1, dW2,
    dtau (sums over its B slices) are compared with the oracle run on those
    slices: Frobenius norms (T3) and row by row (check_grad_rows)."""
    wl = W.WORKLOADS[name]
    x = W.generate(wl)
    heads = [0, wl.H - 1]
    Q, K = x.f64("Q"), x.f64("K")
    keep = np.zeros((wl.B, wl.H, wl.N), bool)
    kaps = {}
    for h in heads:
        W2h = None if x.W2 is None else x.W2[h:h + 1]
        for b in range(wl.B):
            kap = orc.conditioning(Q[b:b + 1, h:h + 1], K[b:b + 1, h:h + 1], x.W1[h:h + 1], W2h,
                                   x.tau[h:h + 1], wl.variant, wl.causal)[0, 0]
            kaps[b, h] = kap
            keep[b, h] = kap <= KAPPA_MAX[wl.io]
    # heads that are not checked keep their full dO (their gradients are not compared)
    others = np.ones(wl.H, bool)
    others[heads] = False
    keep[:, others] = True
    x.dO = x.dO * keep[..., None].astype(x.dO.dtype)
    got_all = gpu_fwd_bwd(F, wl, x, reuse=True)
    dO = x.f64("dO")
    for h in heads:
        refs = [_slice_bwd_oracle(wl, x, b, h) for b in range(wl.B)]
        ref, got = {}, {}
        for n in ("dQ", "dK", "dV"):
            ref[n] = np.concatenate([r[n] for r in refs], axis=0)
            got[n] = got_all[n][:, h:h + 1]
        for n in ("dW1", "dW2", "dtau"):
            if refs[0][n] is None:
                continue
            ref[n] = sum(r[n] for r in refs)
            got[n] = got_all[n][h:h + 1]
        check_grads(wl.io, got, ref, names_of(wl), {"dtau": np.array([sum(r["tau_scale"] for r in refs)])})
        # row-wise, slice by slice
        W2h = None if x.W2 is None else x.W2[h:h + 1]
        for b, r in enumerate(refs):
            sl = (slice(b, b + 1), slice(h, h + 1))
            pq = orc.feature_map(Q[sl], x.W1[h:h + 1], W2h, x.tau[h:h + 1], wl.variant)
            pk = orc.feature_map(K[sl], x.W1[h:h + 1], W2h, x.tau[h:h + 1], wl.variant)
            sc = dv_row_scale(pq, pk, dO[sl], r["den"], kaps[b, h][None, None], wl.causal)
            check_grad_rows(wl.io, {n: got[n][b:b + 1] for n in ("dQ", "dK", "dV")}, r,
                            dv_scale=sc, n_terms=wl.N)
