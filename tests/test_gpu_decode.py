"""GPU parity of the recurrent decode step (flex_decode_step) through the C
ABI: N steps from a zero state against the float64 oracle's causal attention
(forward criteria of tests/parity.py), and the final state against the oracle's
state sum_j phi(K_j)[V_j ; 1]^T."""
import numpy as np
import pytest

import oracle as orc
import workloads as W
from tests.gpu_util import to_device, to_f64
from tests.parity import check_forward, UNIT

pytestmark = pytest.mark.gpu

CASES = [("bf16", 64, 128, "nonstationary"), ("bf16", 32, 64, "stationary"),
         ("f32", 32, 64, "nonstationary"), ("bf16", 128, 256, "nonstationary")]


@pytest.fixture(scope="module")
def F():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_27748_amd as F
    F.load()
    return F


@pytest.mark.parametrize("io,d,m,variant,dv", [c + (c[1],) for c in CASES] +
                         [("bf16", 64, 128, "nonstationary", 32), ("bf16", 32, 64, "stationary", 128),
                          ("f32", 32, 64, "nonstationary", 96)])
def test_decode_steps(F, io, d, m, variant, dv):
    import torch
    wl = W.Workload("decode", 2, 3, 48, d, m, variant, True, io, False, 41, value_dim=dv)
    x = W.generate(wl)
    t = to_device(x)
    desc = F.make_desc(wl.B, wl.H, 1, d, m, variant, True, io, dv=dv)
    state = F.decode_state(desc)
    outs, dens = [], []
    for i in range(wl.N):
        o, den = F.flex_decode_step(desc, t["Q"][:, :, i].contiguous(), t["K"][:, :, i].contiguous(),
                                    t["V"][:, :, i].contiguous(), t["W1"], t["W2"], t["tau"], state)
        outs.append(o)
        dens.append(den)
    O = torch.stack(outs, dim=2)
    den = torch.stack(dens, dim=2)
    torch.cuda.synchronize()
    Q, K, V = x.f64("Q"), x.f64("K"), x.f64("V")
    ref_O, ref_den = orc.linattn_fwd(Q, K, V, x.W1, x.W2, x.tau, variant, True)
    kap = orc.conditioning(Q, K, x.W1, x.W2, x.tau, variant, True)
    check_forward(io, to_f64(O), to_f64(den), ref_O, ref_den, kap)
    # the state: fp32 features and fp32 sums of 48 terms
    pk = orc.feature_map(K, x.W1, x.W2, x.tau, variant)
    Vp = np.concatenate([V, np.ones(V.shape[:-1] + (1,))], axis=-1)
    ref_S = np.einsum("bhnf,bhnv->bhfv", pk, Vp)
    S, z = F.decode_state_views(desc, state)
    got_S = np.concatenate([to_f64(S), to_f64(z)[..., None]], axis=-1)
    err = np.linalg.norm(got_S - ref_S) / np.linalg.norm(ref_S)
    assert err < 2e-5, err


def test_decode_rejects_bad_arguments(F):
    import torch
    desc = F.make_desc(1, 1, 1, 96 + 2, 64, "stationary", True, "bf16")   # d not a multiple of 4
    x = torch.zeros(1, 1, 98, dtype=torch.bfloat16, device="cuda")
    W1 = torch.zeros(1, 64, 98, device="cuda")
    tau = torch.zeros(1, device="cuda")
    st = torch.zeros(1, 1, 128, 99, device="cuda")
    with pytest.raises(F.FlexError):
        F.flex_decode_step(desc, x, x, x, W1, None, tau, st)
    desc = F.make_desc(1, 1, 1, 64, 64, "nonstationary", True, "bf16")   # W2 missing
    x = torch.zeros(1, 1, 64, dtype=torch.bfloat16, device="cuda")
    W1 = torch.zeros(1, 64, 64, device="cuda")
    st = torch.zeros(1, 1, 128, 65, device="cuda")
    with pytest.raises(F.FlexError):
        F.flex_decode_step(desc, x, x, x, W1, None, tau, st)
    W2 = torch.zeros(1, 64, 64, device="cuda")
    with pytest.raises(F.FlexError):                                     # state too small
        F.flex_decode_step(desc, x, x, x, W1, W2, tau, st[..., :64])


def test_decode_state_layout(F):
    """One step from a zero state: S = phi(k) v^T and z = phi(k) land in the
    documented halves of each slice (S rows first, then z)."""
    import torch
    wl = W.Workload("decode1", 2, 2, 1, 32, 64, "stationary", True, "f32", False, 5)
    x = W.generate(wl)
    t = to_device(x)
    desc = F.make_desc(wl.B, wl.H, 1, 32, 64, "stationary", True, "f32")
    state = F.decode_state(desc)
    F.flex_decode_step(desc, t["Q"][:, :, 0].contiguous(), t["K"][:, :, 0].contiguous(),
                       t["V"][:, :, 0].contiguous(), t["W1"], None, t["tau"], state)
    torch.cuda.synchronize()
    pk = orc.feature_map(x.f64("K")[:, :, :1], x.W1, None, x.tau, "stationary")[:, :, 0]
    flat = to_f64(state)
    Fm = 2 * 64
    S = flat[..., :Fm * 32].reshape(2, 2, Fm, 32)
    z = flat[..., Fm * 32:]
    ref_S = pk[..., :, None] * x.f64("V")[:, :, 0][..., None, :]
    assert np.linalg.norm(S - ref_S) <= 1e-5 * np.linalg.norm(ref_S)
    assert np.linalg.norm(z - pk) <= 1e-5 * np.linalg.norm(pk)


PREFILL_CASES = [("bf16", 64, 128, "nonstationary", 0), ("bf16", 64, 128, "nonstationary", 16),
                 ("bf16", 32, 64, "stationary", 32), ("f32", 32, 64, "stationary", 0),
                 ("f32", 32, 64, "nonstationary", 16), ("bf16", 128, 256, "nonstationary", 0),
                 # a padded first frequency group (its padding rows are not state rows)
                 ("bf16", 64, 80, "nonstationary", 0)]
# value widths other than d: the padded run's state keeps the caller's columns
PREFILL_DV_CASES = [("bf16", 64, 128, "nonstationary", 0, 32), ("bf16", 128, 64, "stationary", 16, 64),
                    ("bf16", 32, 80, "nonstationary", 0, 128)]


@pytest.mark.parametrize("io,d,m,variant,chunk,dv", [c + (c[1],) for c in PREFILL_CASES] + PREFILL_DV_CASES)
def test_prefill_then_decode(F, io, d, m, variant, chunk, dv):
    """Prefill a causal prefix of N0 = 300 tokens (3 segments), then decode 6
    more tokens from the prefill's state.  The prefill's O and den are bitwise
    those of flex_linattn_fwd; its state is sum_j phi(K_j) [V_j ; 1]^T over the
    prefix (within the rounding of the features it sums); the decode outputs
    are rows N0 .. N0+5 of the oracle's causal attention over all 306 tokens."""
    import torch
    N0, steps = 300, 6
    wl = W.Workload("prefill", 2, 3, N0 + steps, d, m, variant, True, io, False, 43, value_dim=dv)
    x = W.generate(wl)
    t = to_device(x)
    pre = {k: t[k][:, :, :N0].contiguous() for k in ("Q", "K", "V")}
    dp = F.make_desc(wl.B, wl.H, N0, d, m, variant, True, io, dv=dv, segments=3, chunk=chunk)
    O_p, den_p, state = F.flex_linattn_prefill(dp, pre["Q"], pre["K"], pre["V"], t["W1"], t["W2"],
                                               t["tau"])
    O_f, den_f = F.flex_linattn_fwd(dp, pre["Q"], pre["K"], pre["V"], t["W1"], t["W2"], t["tau"])
    torch.cuda.synchronize()
    assert torch.equal(O_p.view(torch.int16) if io == "bf16" else O_p,
                       O_f.view(torch.int16) if io == "bf16" else O_f)
    assert torch.equal(den_p, den_f)
    # the prefill state against the oracle's prefix sum, relative to the
    # magnitude of the summed terms (features rounded to the io precision,
    # fp32 accumulation over N0 terms)
    Q, K, V = x.f64("Q"), x.f64("K"), x.f64("V")
    pk = orc.feature_map(K[:, :, :N0], x.W1, x.W2, x.tau, variant)
    Vp = np.concatenate([V[:, :, :N0], np.ones(V[:, :, :N0].shape[:-1] + (1,))], axis=-1)
    ref_S = np.einsum("bhnf,bhnv->bhfv", pk, Vp)
    abs_S = np.einsum("bhnf,bhnv->bhfv", np.abs(pk), np.abs(Vp))
    S, z = F.decode_state_views(dp, state)
    got_S = np.concatenate([to_f64(S), to_f64(z)[..., None]], axis=-1)
    bound = (4 * UNIT[io] + 4 * 2.0 ** -24 * np.sqrt(N0)) * np.linalg.norm(abs_S)
    assert np.linalg.norm(got_S - ref_S) <= bound, (np.linalg.norm(got_S - ref_S), bound)
    # decode the next tokens from the prefill's state
    dd = F.make_desc(wl.B, wl.H, 1, d, m, variant, True, io, dv=dv)
    outs, dens = [], []
    for i in range(N0, N0 + steps):
        o, den = F.flex_decode_step(dd, t["Q"][:, :, i].contiguous(), t["K"][:, :, i].contiguous(),
                                    t["V"][:, :, i].contiguous(), t["W1"], t["W2"], t["tau"], state)
        outs.append(o)
        dens.append(den)
    O = torch.stack(outs, dim=2)
    den = torch.stack(dens, dim=2)
    torch.cuda.synchronize()
    ref_O, ref_den = orc.linattn_fwd(Q, K, V, x.W1, x.W2, x.tau, variant, True)
    kap = orc.conditioning(Q, K, x.W1, x.W2, x.tau, variant, True)
    check_forward(io, to_f64(O), to_f64(den), ref_O[:, :, N0:], ref_den[:, :, N0:], kap[:, :, N0:])


def test_prefill_rejects_non_causal_and_missing_state(F):
    import torch
    d = F.make_desc(1, 2, 64, 64, 64, "stationary", False, "bf16")
    x = torch.zeros(1, 2, 64, 64, dtype=torch.bfloat16, device="cuda")
    W1 = torch.zeros(2, 64, 64, device="cuda")
    tau = torch.zeros(2, device="cuda")
    with pytest.raises(F.FlexError) as e:
        F.flex_linattn_prefill(d, x, x, x, W1, None, tau)
    assert e.value.status == F.FLEX_ERR_UNSUPPORTED
