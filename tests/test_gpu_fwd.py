"""GPU parity of the feature map and the forward pass against the float64 oracle.

All calls go through the C ABI of libflexattn.so.  Inputs are the seeded
synthetic workloads; small cases span several 64-token chunks plus a ragged
tail, full-size cases check sampled rows in the launch configuration the
benchmark times.
"""
import math

import numpy as np
import pytest

import oracle as orc
import workloads as W
from tests.gpu_util import to_device, to_f64, desc_of
from tests.parity import check_forward, abs_scales, TOL, UNIT

pytestmark = pytest.mark.gpu

SHAPES = [  # (io, d, m)
    ("f32", 32, 64), ("bf16", 32, 64), ("bf16", 64, 64), ("bf16", 64, 128), ("bf16", 128, 256),
]
# attention shapes that run as frequency groups of 64 (besides d = 128, m = 256)
GROUP_SHAPES = [("f32", 32, 128), ("bf16", 32, 192), ("bf16", 64, 256), ("bf16", 128, 64), ("bf16", 128, 128),
                # a last group that 64 does not fill (zero-padded rows, masked features)
                ("bf16", 32, 16), ("bf16", 64, 48), ("bf16", 128, 80), ("f32", 32, 96)]


@pytest.fixture(scope="module")
def F():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_27748_amd as F
    F.load()
    return F


def small(io, d, m, variant, causal, B=2, H=3, N=200, seed=7):
    wl = W.Workload("small", B, H, N, d, m, variant, causal, io, True, seed)
    return wl, W.generate(wl)


def oracle_fwd(x, wl):
    O, den = orc.linattn_fwd(x.f64("Q"), x.f64("K"), x.f64("V"), x.W1, x.W2, x.tau,
                             wl.variant, wl.causal)
    kap = orc.conditioning(x.f64("Q"), x.f64("K"), x.W1, x.W2, x.tau, wl.variant, wl.causal)
    return O, den, kap, abs_scales(x, wl)


@pytest.mark.parametrize("io,d,m", SHAPES + GROUP_SHAPES)
@pytest.mark.parametrize("variant", ["stationary", "nonstationary"])
def test_feature_map(F, io, d, m, variant):
    wl, x = small(io, d, m, variant, False, N=131)
    t = to_device(x)
    Phi = F.flex_feature_map(desc_of(wl), t["Q"], t["W1"], t["W2"], t["tau"])
    got = to_f64(Phi)
    ref = orc.feature_map(x.f64("Q"), x.W1, x.W2, x.tau, variant)
    # |phi| <= s e(x): compare relative to that row scale
    s = 1 / math.sqrt(m) if variant == "stationary" else 1 / (2 * math.sqrt(m))
    scale = s * orc.norm_factor(x.f64("Q"), x.tau)[..., None]
    err = np.max(np.abs(got - ref) / scale)
    # fp32: phase and norm factor in float64, features rounded to fp32 about
    # twice (a few units of 2^-24); bf16: one rounding of the stored value
    tol = 1e-6 if io == "f32" else 2.0 ** -8
    assert err <= tol, err


@pytest.mark.parametrize("variant", ["stationary", "nonstationary"])
def test_feature_map_several_chunks_per_workgroup(F, variant):
    """Enough chunks (8 x 8 slices x 24) that each workgroup maps several in
    turn, prefetching the next one; N = 1500 leaves a ragged last chunk."""
    wl = W.Workload("fmap_many", 8, 8, 1500, 64, 64, variant, False, "bf16", True, 17)
    x = W.generate(wl)
    t = to_device(x)
    Phi = F.flex_feature_map(desc_of(wl), t["Q"], t["W1"], t["W2"], t["tau"])
    got = to_f64(Phi)
    ref = orc.feature_map(x.f64("Q"), x.W1, x.W2, x.tau, variant)
    s = 1 / math.sqrt(wl.m) if variant == "stationary" else 1 / (2 * math.sqrt(wl.m))
    scale = s * orc.norm_factor(x.f64("Q"), x.tau)[..., None]
    assert np.max(np.abs(got - ref) / scale) <= 2.0 ** -8


@pytest.mark.parametrize("io,d,m", SHAPES + GROUP_SHAPES)
@pytest.mark.parametrize("variant", ["stationary", "nonstationary"])
@pytest.mark.parametrize("causal", [False, True])
def test_forward_small(F, io, d, m, variant, causal):
    wl, x = small(io, d, m, variant, causal)
    t = to_device(x)
    O, den = F.flex_linattn_fwd(desc_of(wl), t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"])
    O_ref, den_ref, kap, sc = oracle_fwd(x, wl)
    check_forward(io, to_f64(O), to_f64(den), O_ref, den_ref, kap, sc)


# (d, d_v) with d_v != d: run at width max(d, d_v) on zero-padded copies
VALUE_WIDTHS = [(64, 32), (128, 64), (128, 32), (32, 64), (64, 128), (32, 128)]


@pytest.mark.parametrize("d,dv", VALUE_WIDTHS)
@pytest.mark.parametrize("variant", ["stationary", "nonstationary"])
@pytest.mark.parametrize("causal", [False, True])
def test_forward_value_width(F, d, dv, variant, causal):
    import torch
    wl = W.Workload("dv", 2, 2, 150, d, 80, variant, causal, "bf16", False, 61, value_dim=dv)
    x = W.generate(wl)
    t = to_device(x)
    O, den = F.flex_linattn_fwd(desc_of(wl), t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"])
    assert tuple(O.shape) == (2, 2, 150, dv)
    O_ref, den_ref, kap, sc = oracle_fwd(x, wl)
    check_forward("bf16", to_f64(O), to_f64(den), O_ref, den_ref, kap, sc)
    # the allocation-free entry point takes the same route (its scratch holds
    # the padded copies at this size): the same bits
    O2, den2 = torch.empty_like(O), torch.empty_like(den)
    F.flex_linattn_fwd_noalloc(desc_of(wl), t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"], O2, den2)
    assert torch.equal(O2.view(torch.int16), O.view(torch.int16))
    assert torch.equal(den2.view(torch.int32), den.view(torch.int32))


@pytest.mark.parametrize("causal", [False, True])
def test_forward_many_segments(F, causal):
    """20 segments: the segment scan takes its states in two batches."""
    wl, x = small("bf16", 64, 64, "nonstationary", causal, B=1, H=2, N=1350, seed=13)
    t = to_device(x)
    O, den = F.flex_linattn_fwd(desc_of(wl, segments=20), t["Q"], t["K"], t["V"],
                                t["W1"], t["W2"], t["tau"])
    O_ref, den_ref, kap, sc = oracle_fwd(x, wl)
    check_forward("bf16", to_f64(O), to_f64(den), O_ref, den_ref, kap, sc)


@pytest.mark.parametrize("segments", [1, 2, 3, 5])
@pytest.mark.parametrize("causal", [False, True])
def test_forward_segments(F, segments, causal):
    """The result does not depend on how the sequence is split into segments
    (state carried across workgroups by the segment scan)."""
    wl, x = small("bf16", 64, 128, "nonstationary", causal, B=1, H=2, N=330, seed=11)
    t = to_device(x)
    O, den = F.flex_linattn_fwd(desc_of(wl, segments=segments), t["Q"], t["K"], t["V"],
                                t["W1"], t["W2"], t["tau"])
    O_ref, den_ref, kap, sc = oracle_fwd(x, wl)
    check_forward("bf16", to_f64(O), to_f64(den), O_ref, den_ref, kap, sc)


@pytest.mark.parametrize("N", [1, 2, 63, 64, 65, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_forward_edge_lengths(F, N, causal):
    wl, x = small("bf16", 64, 64, "stationary", causal, B=1, H=2, N=N, seed=13)
    t = to_device(x)
    O, den = F.flex_linattn_fwd(desc_of(wl), t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"])
    O_ref, den_ref, kap, sc = oracle_fwd(x, wl)
    check_forward("bf16", to_f64(O), to_f64(den), O_ref, den_ref, kap, sc)
    if causal:
        # a token attends only to itself at i = 0: O_0 = V_0 up to the output rounding
        np.testing.assert_allclose(to_f64(O)[:, :, 0], x.f64("V")[:, :, 0], rtol=2 ** -8, atol=1e-6)


@pytest.mark.parametrize("io,d,m", SHAPES)
@pytest.mark.parametrize("variant", ["stationary", "nonstationary"])
def test_forward_chunk_invariance(F, io, d, m, variant):
    """Chunk lengths C = 16, 32, 64 of the causal sweep (tril inside a chunk,
    the running state across chunks) give the same attention: each matches the
    oracle, and any two differ by no more than the rounding of the features
    they contract in a different order.  N = 203 with 3 segments leaves ragged
    last chunks and segment boundaries inside every chunk length's grid."""
    wl, x = small(io, d, m, variant, True, B=1, H=2, N=203, seed=19)
    t = to_device(x)
    O_ref, den_ref, kap, sc = oracle_fwd(x, wl)
    outs = {}
    for C in (16, 32, 64):
        O, den = F.flex_linattn_fwd(desc_of(wl, segments=3, chunk=C), t["Q"], t["K"], t["V"],
                                    t["W1"], t["W2"], t["tau"])
        outs[C] = (to_f64(O), to_f64(den))
        check_forward(io, outs[C][0], outs[C][1], O_ref, den_ref, kap, sc)
    # den: the same sums grouped differently (intra-chunk products rounded to
    # the feature type, or the carried state rounded to it).  Either rounding
    # moves a row by at most u/2 of sum_j sum_f |phi(Q_i)_f phi(K_j)_f| (T1a's
    # scale); fp32 adds the accumulation order over up to 203 terms.
    den_abs = sc[1]
    bound = (4 if io == "bf16" else 64) * UNIT[io]
    for a, b in ((16, 32), (16, 64), (32, 64)):
        diff = np.abs(outs[a][1] - outs[b][1]) / den_abs
        assert np.max(diff) <= bound, (a, b, np.max(diff))


def test_forward_deterministic_and_den_optional(F):
    import torch
    wl, x = small("bf16", 64, 128, "nonstationary", True, N=300)
    t = to_device(x)
    d = desc_of(wl)
    O1, den1 = F.flex_linattn_fwd(d, t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"])
    O2, den2 = F.flex_linattn_fwd(d, t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"])
    O3, den3 = F.flex_linattn_fwd(d, t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"],
                                  want_den=False)
    torch.cuda.synchronize()
    assert den3 is None
    assert torch.equal(O1.view(torch.int16), O2.view(torch.int16))
    assert torch.equal(den1, den2)
    assert torch.equal(O1.view(torch.int16), O3.view(torch.int16))


def test_forward_sigma_invariance(F):
    """O does not depend on sigma (it scales phi); den scales by sigma^2."""
    wl, x = small("f32", 32, 64, "stationary", True, N=150)
    t = to_device(x)
    O1, d1 = F.flex_linattn_fwd(desc_of(wl), t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"])
    O2, d2 = F.flex_linattn_fwd(desc_of(wl, sigma=2.0), t["Q"], t["K"], t["V"], t["W1"], t["W2"],
                                t["tau"])
    np.testing.assert_allclose(to_f64(d2), 4 * to_f64(d1), rtol=1e-6)
    np.testing.assert_array_equal(to_f64(O1), to_f64(O2))


FULL_FWD = ["tiny_stationary_noncausal_f32", "lm_stationary_causal", "long_stationary_noncausal",
            "nonstationary_causal_train", "train_at_scale_d128", "headline_causal_train_d64"]


def _check_sampled_rows(wl, x, O, den, rows, kappa=None, ref=None):
    """Sampled rows of a GPU forward (O, den as float64 arrays) against the
    oracle's per-row definition, with the T1/T2 reading of the parity tests.
    kappa: the oracle's condition numbers of the whole input, and ref: the
    oracle's (O, den) of the rows, if already computed."""
    rows = np.array(rows)
    Q, K, V = x.f64("Q"), x.f64("K"), x.f64("V")
    O_ref, den_ref = ref if ref is not None else orc.linattn_fwd_rows(Q, K, V, x.W1, x.W2, x.tau, wl.variant,
                                                                      wl.causal, rows)
    # conditioning of the sampled rows
    kap = np.empty(len(rows))
    for r, (b, h, i) in enumerate(rows):
        if kappa is not None:
            kap[r] = kappa[b, h, i]
            continue
        sl = slice(None, i + 1) if wl.causal else slice(None)
        Wb = None if x.W2 is None else x.W2[h:h + 1]
        pq = orc.feature_map(Q[b:b + 1, h:h + 1, i:i + 1], x.W1[h:h + 1], Wb, x.tau[h:h + 1], wl.variant)
        pk = orc.feature_map(K[b:b + 1, h:h + 1, sl], x.W1[h:h + 1], Wb, x.tau[h:h + 1], wl.variant)
        tq = pq[0, 0, 0] * pk[0, 0].sum(0)
        kap[r] = np.abs(tq).sum() / abs(tq.sum())
    got_O = O[rows[:, 0], rows[:, 1], rows[:, 2]]
    got_den = den[rows[:, 0], rows[:, 1], rows[:, 2]]
    tol = TOL[wl.io]
    rel_den = np.linalg.norm(got_den - den_ref) / np.linalg.norm(den_ref)
    num_g = got_O * got_den[:, None]
    num_r = O_ref * den_ref[:, None]
    rel_num = np.linalg.norm(num_g - num_r) / np.linalg.norm(num_r)
    assert rel_den <= tol and rel_num <= tol, (rel_den, rel_num)
    keep = kap <= (1e3 if wl.io == "f32" else 20.0)
    if keep.any():
        rel_O = np.linalg.norm(got_O[keep] - O_ref[keep]) / np.linalg.norm(O_ref[keep])
        assert rel_O <= tol, rel_O
    assert np.all(np.isfinite(O[..., 0]) | (den == 0))


@pytest.mark.parametrize("name", FULL_FWD)
def test_forward_full_size_sampled(F, name):
    """Full configured sizes, default launch configuration; rows sampled across
    slices, chunk boundaries, segment boundaries and the sequence end are
    compared with the oracle's per-row definition."""
    wl = W.WORKLOADS[name]
    x = W.generate(wl, with_grad=False)
    t = to_device(x)
    O, den = F.flex_linattn_fwd(desc_of(wl), t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"])
    O = to_f64(O)
    den = to_f64(den)
    # every (b,h) slice: two random rows and one boundary row (chunk, segment
    # or sequence end), so a mapping error confined to some slices is seen
    rng = np.random.default_rng(5)
    idx = [0, 1, 63, 64, 65, wl.N // 2, wl.N - 65, wl.N - 1]
    rows = []
    for b in range(wl.B):
        for h in range(wl.H):
            for i in list(rng.integers(0, wl.N, 2)) + ([idx[(b * wl.H + h) % len(idx)]]):
                rows.append((b, h, int(i)))
    _check_sampled_rows(wl, x, O, den, rows)


@pytest.fixture(scope="module")
def long_input():
    """A long ragged sequence over few heads (B*H = 2, N = 65573: 1025 chunks,
    the last one of 37 tokens), its sampled rows (chunk and segment boundaries,
    the sequence end, random positions) and the oracle's values there."""
    wl = W.Workload("long_few_heads", 1, 2, 65573, 64, 128, "nonstationary", True, "bf16", False, 47)
    x = W.generate(wl, with_grad=False)
    kappa = orc.conditioning(x.f64("Q"), x.f64("K"), x.W1, x.W2, x.tau, wl.variant, wl.causal)
    rng = np.random.default_rng(11)
    seg = 5 * 64   # tokens per segment at 256 segments
    idx = [0, 63, 64, seg - 1, seg, 204 * seg - 1, 204 * seg, 8 * 64 - 1, 8 * 64, wl.N - 38, wl.N - 37,
           wl.N - 1]
    rows = [(0, h, int(i)) for h in range(wl.H) for i in idx + list(rng.integers(0, wl.N, 3))]
    ref = orc.linattn_fwd_rows(x.f64("Q"), x.f64("K"), x.f64("V"), x.W1, x.W2, x.tau, wl.variant, wl.causal,
                               np.array(rows))
    return wl, x, kappa, rows, ref


@pytest.mark.parametrize("segments", [0, 256])
def test_forward_long_sequence_sampled(F, long_input, segments):
    """The long input with the heuristic's segment count and with 256 segments
    of 5 chunks (205 hold chunks, the 51 trailing ones are empty)."""
    wl, x, kappa, rows, ref = long_input
    t = to_device(x)
    O, den = F.flex_linattn_fwd(desc_of(wl, segments=segments), t["Q"], t["K"], t["V"], t["W1"], t["W2"],
                                t["tau"])
    _check_sampled_rows(wl, x, to_f64(O), to_f64(den), rows, kappa, ref)
