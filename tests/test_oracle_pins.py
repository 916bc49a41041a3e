"""Pins of the float64 oracle against what the paper and the mathematics fix.

Each test names the passage it follows.  None compares the oracle with itself:
they use closed forms, Monte-Carlo limits of the kernels the frequency laws
imply, brute force (the quadratic form of Eq.(attention)), special cases and
central finite differences.
"""
import math

import numpy as np
import pytest

import oracle as orc

S, NS = orc.STATIONARY, orc.NONSTATIONARY


def _rng(seed):
    return np.random.default_rng(seed)


def _small_inputs(variant, seed=0, B=2, H=2, N=9, d=5, m=6, scale=0.6, dv=None):
    r = _rng(seed)
    W1 = r.standard_normal((H, m, d))
    W2 = r.standard_normal((H, m, d)) if variant == NS else None
    Q = r.standard_normal((B, H, N, d)) * scale
    K = r.standard_normal((B, H, N, d)) * scale
    V = r.standard_normal((B, H, N, d if dv is None else dv))
    tau = np.array([math.log(2.0), 0.9])[:H]
    return Q, K, V, W1, W2, tau


# --- closed forms of the feature map (Eq.(phi_n), Eq.(phi_non), norm factor) ----

def test_stationary_feature_closed_form():
    """W = identity rows, x = (pi/3, pi/2, 0): cos/sin values are exact; the
    [cos block | sin block] order and s = sigma/sqrt(m) are as printed
    (Sec. 3.1, phi_n), with the norm factor exp(||x||^2/exp(tau))."""
    d = 3
    W = np.eye(d)[None]                     # m = d = 3 frequencies e_1, e_2, e_3
    x = np.array([math.pi / 3, math.pi / 2, 0.0])
    tau = np.array([math.log(5.0)])
    sigma = 1.7
    phi = orc.feature_map(x[None, None, None], W, None, tau, S, sigma)[0, 0, 0]
    e = math.exp((math.pi ** 2 / 9 + math.pi ** 2 / 4) / 5.0)
    want = sigma / math.sqrt(3) * e * np.array([0.5, 0.0, 1.0, math.sqrt(3) / 2, 1.0, 0.0])
    np.testing.assert_allclose(phi, want, rtol=1e-14, atol=1e-14)


def test_nonstationary_feature_closed_form():
    """omega'_1 = (w1+w2)/2, omega'_2 = (w1-w2)/2 and
    phi = sigma/(2 sqrt(m)) e(x) [cos P1 cos P2 | sin P1 cos P2] (Sec. 3.2)."""
    W1 = np.array([[[1.0, 1.0]]])           # m = 1, d = 2
    W2 = np.array([[[1.0, -1.0]]])
    # W'1 = (1, 0), W'2 = (0, 1); x = (pi/6, pi/3): P1 = pi/6, P2 = pi/3
    x = np.array([math.pi / 6, math.pi / 3])
    tau = np.array([math.inf])              # norm factor exactly 1
    phi = orc.feature_map(x[None, None, None], W1, W2, tau, NS, 1.0)[0, 0, 0]
    want = 0.5 * np.array([math.sqrt(3) / 2 * 0.5, 0.5 * 0.5])
    np.testing.assert_allclose(phi, want, rtol=1e-14, atol=1e-15)


def test_sum_to_product_identity():
    """C5: cos a + cos b = 2 cos P1 cos P2 and sin a + sin b = 2 sin P1 cos P2
    with a = w1.x, b = w2.x (the step inside Eq.(phi_non))."""
    r = _rng(5)
    W1 = r.standard_normal((2, 16, 7))
    W2 = r.standard_normal((2, 16, 7))
    X = r.standard_normal((3, 2, 11, 7))
    tau = np.array([0.3, -0.2])
    phi = orc.feature_map(X, W1, W2, tau, NS, 1.0)
    a = np.matmul(X, np.swapaxes(W1, -1, -2)[None])
    b = np.matmul(X, np.swapaxes(W2, -1, -2)[None])
    e = np.exp((X * X).sum(-1) / np.exp(tau)[None, :, None])[..., None]
    s = 1.0 / (2 * math.sqrt(16))
    want = s * e * 0.5 * np.concatenate([np.cos(a) + np.cos(b), np.sin(a) + np.sin(b)], -1)
    np.testing.assert_allclose(phi, want, rtol=1e-12, atol=1e-13)


# --- Monte-Carlo limits of the kernels (Bochner / Yaglom, Sec. 3.1-3.2) -------------

def _pairs(d, n, scale, seed):
    r = _rng(seed)
    x = r.standard_normal((n, d)) * scale
    y = r.standard_normal((n, d)) * scale
    return x, y


def _kernel_estimates(variant, W1, W2, tau, x, y, sigma=1.0):
    X = np.concatenate([x, y])[None, None]
    phi = orc.feature_map(X, W1, W2, tau, variant, sigma)[0, 0]
    n = len(x)
    return np.sum(phi[:n] * phi[n:], axis=-1)


@pytest.mark.parametrize("sigma", [1.0, 1.5])
def test_stationary_mc_gaussian_kernel(sigma):
    """C2: omega ~ N(0, I), no norm factor => phi(x).phi(y) -> sigma^2 exp(-|x-y|^2/2)
    (Bochner, Thm 3.1 and Eq.(phi_n)); the error shrinks like m^-1/2."""
    d = 4
    x, y = _pairs(d, 64, 0.5, 1)
    want = sigma ** 2 * np.exp(-0.5 * np.sum((x - y) ** 2, -1))
    errs = []
    for m, seed in [(64, 2), (2 ** 16, 3)]:
        W = _rng(seed).standard_normal((1, m, d))
        est = _kernel_estimates(S, W, None, np.array([math.inf]), x, y, sigma)
        errs.append(np.mean(np.abs(est - want)))
    assert errs[1] < 4.0 * sigma ** 2 / math.sqrt(2 ** 16)
    assert errs[0] > 4 * errs[1]


def test_softmax_recovery_mc():
    """C3: with the norm factor c = 2 (2 sqrt(d) in units where x carries d^-1/4),
    phi~(x).phi~(y) -> exp(x.y) (Eq.(softmax kernel) and the RFA feature map)."""
    d = 4
    x, y = _pairs(d, 64, 0.4, 11)
    want = np.exp(np.sum(x * y, -1))
    m = 2 ** 16
    W = _rng(12).standard_normal((1, m, d))
    est = _kernel_estimates(S, W, None, np.array([math.log(2.0)]), x, y)
    assert np.mean(np.abs(est - want) / want) < 4.0 / math.sqrt(m) * 3


def test_nonstationary_mc_kernel():
    """C4: omega_1, omega_2 iid N(0, I): the expectation in Eq.(phi_non) is
    k(x,y) = (sigma^2/2)[exp(-|x-y|^2/2) + exp(-(|x|^2+|y|^2)/2)]; the printed
    phi (scale sigma/(2 sqrt(n))) estimates k/4 (see DESIGN readings)."""
    d = 4
    sigma = 1.3
    x, y = _pairs(d, 64, 0.6, 21)
    k = sigma ** 2 / 2 * (np.exp(-0.5 * np.sum((x - y) ** 2, -1))
                          + np.exp(-0.5 * (np.sum(x * x, -1) + np.sum(y * y, -1))))
    m = 2 ** 16
    r = _rng(22)
    W1 = r.standard_normal((1, m, d))
    W2 = r.standard_normal((1, m, d))
    est = _kernel_estimates(NS, W1, W2, np.array([math.inf]), x, y, sigma)
    assert np.mean(np.abs(est - k / 4)) < 4.0 * sigma ** 2 / math.sqrt(m)
    # and clearly not k itself
    assert np.mean(np.abs(est - k)) > 0.3


# --- attention: brute force and special cases (Eq.(attention), Eq.(linear att)) ---

def _quadratic(Q, K, V, W1, W2, tau, variant, causal, sigma=1.0):
    """Eq.(attention) with sim(q,k) = phi~(q).phi~(k), the N x N way."""
    pq = orc.feature_map(Q, W1, W2, tau, variant, sigma)
    pk = orc.feature_map(K, W1, W2, tau, variant, sigma)
    A = np.matmul(pq, np.swapaxes(pk, -1, -2))
    if causal:
        A = np.tril(A)
    num = np.matmul(A, V)
    den = A.sum(-1)
    return num / den[..., None], den, A


@pytest.mark.parametrize("variant", [S, NS])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("dv", [None, 2, 8])
def test_state_form_equals_quadratic(variant, causal, dv):
    """C1: the state form equals the quadratic form (exactness of Eq.(linear att)),
    also with a value width other than d."""
    Q, K, V, W1, W2, tau = _small_inputs(variant, seed=3, dv=dv)
    O, den = orc.linattn_fwd(Q, K, V, W1, W2, tau, variant, causal)
    Oq, denq, _ = _quadratic(Q, K, V, W1, W2, tau, variant, causal)
    np.testing.assert_allclose(den, denq, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(O * den[..., None], Oq * denq[..., None], rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("variant", [S, NS])
def test_decode_steps_equal_causal_quadratic(variant):
    """Recurrent decode (Sec. 4.2's autoregressive use of Eq.(linear att)): t
    steps from a zero state give row t of the causal brute-force attention, and
    the state is the plain sum of phi(k_j)[v_j ; 1]^T over the prefix."""
    Q, K, V, W1, W2, tau = _small_inputs(variant, seed=5, N=11)
    Oq, denq, _ = _quadratic(Q, K, V, W1, W2, tau, variant, True)
    B, H, N, d = Q.shape
    m = W1.shape[1]
    state = np.zeros((B, H, 2 * m, d + 1))
    for t in range(N):
        o, den, state = orc.decode_step(state, Q[:, :, t], K[:, :, t], V[:, :, t], W1, W2, tau, variant)
        np.testing.assert_allclose(den, denq[:, :, t], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(o * den[..., None], Oq[:, :, t] * denq[:, :, t, None], rtol=1e-11, atol=1e-11)
    pk = orc.feature_map(K, W1, W2, tau, variant)
    Vp = np.concatenate([V, np.ones(V.shape[:-1] + (1,))], axis=-1)
    total = np.einsum("bhnf,bhnv->bhfv", pk, Vp)
    np.testing.assert_allclose(state, total, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_rows_equal_full(causal):
    """The per-row evaluation used for full-size spot checks agrees with the
    full oracle (both are Eq.(linear att); one per row, one for all rows)."""
    Q, K, V, W1, W2, tau = _small_inputs(NS, seed=4)
    O, den = orc.linattn_fwd(Q, K, V, W1, W2, tau, NS, causal)
    rows = np.array([[0, 0, 0], [1, 1, 8], [0, 1, 4], [1, 0, 7]])
    Or, dr = orc.linattn_fwd_rows(Q, K, V, W1, W2, tau, NS, causal, rows)
    for r, (b, h, i) in enumerate(rows):
        np.testing.assert_allclose(dr[r], den[b, h, i], rtol=1e-12)
        np.testing.assert_allclose(Or[r] * dr[r], O[b, h, i] * den[b, h, i], rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("variant", [S, NS])
def test_constant_features_give_means(variant):
    """C6: W = 0 and tau -> inf make every feature vector equal, so causal
    attention is the prefix mean of V and non-causal attention the mean."""
    Q, K, V, W1, W2, tau = _small_inputs(variant, seed=6)
    W1 = np.zeros_like(W1)
    W2 = None if W2 is None else np.zeros_like(W2)
    tau = np.full_like(tau, math.inf)
    O, _ = orc.linattn_fwd(Q, K, V, W1, W2, tau, variant, True)
    want = np.cumsum(V, axis=2) / np.arange(1, V.shape[2] + 1)[None, None, :, None]
    np.testing.assert_allclose(O, want, rtol=1e-13, atol=1e-14)
    O, _ = orc.linattn_fwd(Q, K, V, W1, W2, tau, variant, False)
    np.testing.assert_allclose(O, np.broadcast_to(V.mean(2, keepdims=True), V.shape),
                               rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("variant", [S, NS])
def test_invariances(variant):
    """C7: O does not depend on sigma nor on a positive per-query rescaling of
    phi(Q) (so the query norm factor cancels); causal O_1 = V_1; the last causal
    row equals the last non-causal row."""
    Q, K, V, W1, W2, tau = _small_inputs(variant, seed=7)
    O1, _ = orc.linattn_fwd(Q, K, V, W1, W2, tau, variant, True)
    O2, _ = orc.linattn_fwd(Q, K, V, W1, W2, tau, variant, True, sigma=3.0)
    np.testing.assert_allclose(O1, O2, rtol=1e-9, atol=1e-12)
    pq = orc.feature_map(Q, W1, W2, tau, variant)
    pk = orc.feature_map(K, W1, W2, tau, variant)
    r = _rng(8).uniform(0.1, 10.0, pq.shape[:-1])[..., None]
    n1, d1 = orc.attend_features(pq, pk, V, True)
    n2, d2 = orc.attend_features(pq * r, pk, V, True)
    np.testing.assert_allclose(n1 / d1[..., None], n2 / d2[..., None], rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(O1[:, :, 0], V[:, :, 0], rtol=1e-12)
    On, _ = orc.linattn_fwd(Q, K, V, W1, W2, tau, variant, False)
    np.testing.assert_allclose(O1[:, :, -1] * 1.0, On[:, :, -1], rtol=1e-10, atol=1e-12)


def test_large_m_recovers_softmax_attention():
    """C9: Gaussian frequencies with c = 2 recover softmax attention
    exp(q.k) / sum exp(q.k) as m grows (Sec. 3.2, Flexformer_s with Gaussian
    frequencies is the RFA estimate of the softmax kernel)."""
    r = _rng(9)
    B, H, N, d, m = 1, 1, 12, 4, 2 ** 16
    Q = r.standard_normal((B, H, N, d)) * 0.3
    K = r.standard_normal((B, H, N, d)) * 0.3
    V = r.standard_normal((B, H, N, d))
    W = r.standard_normal((H, m, d))
    tau = np.array([math.log(2.0)])
    for causal in (False, True):
        O, _ = orc.linattn_fwd(Q, K, V, W, None, tau, S, causal)
        A = np.exp(np.matmul(Q, np.swapaxes(K, -1, -2)))
        if causal:
            A = np.tril(A)
        Osm = np.matmul(A, V) / A.sum(-1, keepdims=True)
        assert np.max(np.abs(O - Osm)) < 0.05


def test_conditioning_bounds():
    """kappa_i >= 1, with equality when every term of den_i is positive."""
    Q, K, V, W1, W2, tau = _small_inputs(S, seed=10)
    kap = orc.conditioning(Q, K, W1, None, tau, S, True)
    assert np.all(kap >= 1 - 1e-12)
    kap0 = orc.conditioning(Q, K, np.zeros_like(W1), None, tau, S, True)
    np.testing.assert_allclose(kap0, 1.0, rtol=1e-12)


@pytest.mark.parametrize("variant", [S, NS])
@pytest.mark.parametrize("causal", [False, True])
def test_conditioning_den_is_attention_den(variant, causal):
    """The dot products whose condition numbers kappa_i measures are the
    denominators of Eq.(linear att): phi(Q_i)^T z_i with z_i the sum of phi(K_j)
    over j <= i (causal, inclusive) or over all j.  Their sum must equal the
    quadratic form's row sums (brute force, independent of the state form), so
    an exclusive, shifted or non-cumulative z fails."""
    Q, K, V, W1, W2, tau = _small_inputs(variant, seed=14)
    kap, den = orc.conditioning(Q, K, W1, W2, tau, variant, causal, return_den=True)
    _, denq, _ = _quadratic(Q, K, V, W1, W2, tau, variant, causal)
    np.testing.assert_allclose(den, denq, rtol=1e-12, atol=1e-13)
    assert np.all(kap >= 1 - 1e-12)


def test_conditioning_two_tokens_closed_form():
    """Two tokens, one frequency w = 1, d = 1, tau -> inf (norm factor 1), so
    phi(x) = [cos x, sin x] (Eq.(phi_n) with m = 1, sigma = 1).  Keys k_1 = 0,
    k_2 = pi/2 give phi(k_1) = (1, 0), phi(k_2) = (0, 1); queries q_1 = 5 pi/6,
    q_2 = 2 pi/3.  Causal: z_1 = (1, 0) gives den_1 = -sqrt(3)/2 and kappa_1 = 1;
    z_2 = (1, 1) gives den_2 = -1/2 + sqrt(3)/2 and kappa_2 = (1/2 + sqrt(3)/2) /
    (sqrt(3)/2 - 1/2) = 2 + sqrt(3).  Non-causal: z = (1, 1) for both rows, and
    kappa_1 = (sqrt(3)/2 + 1/2) / (sqrt(3)/2 - 1/2) = 2 + sqrt(3) as well.  An
    exclusive prefix (z_2 = (1, 0)) or a non-cumulative z (z_2 = (0, 1)) would
    give kappa_2 = 1."""
    W = np.ones((1, 1, 1))
    tau = np.array([math.inf])
    Q = np.array([5 * math.pi / 6, 2 * math.pi / 3]).reshape(1, 1, 2, 1)
    K = np.array([0.0, math.pi / 2]).reshape(1, 1, 2, 1)
    r3 = math.sqrt(3.0)
    kap, den = orc.conditioning(Q, K, W, None, tau, S, True, return_den=True)
    np.testing.assert_allclose(den[0, 0], [-r3 / 2, -0.5 + r3 / 2], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(kap[0, 0], [1.0, 2 + r3], rtol=1e-13)
    kap, den = orc.conditioning(Q, K, W, None, tau, S, False, return_den=True)
    np.testing.assert_allclose(den[0, 0], [-r3 / 2 + 0.5, -0.5 + r3 / 2], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(kap[0, 0], [2 + r3, 2 + r3], rtol=1e-13)


# --- backward: closed form in V and finite differences --------------------------------

@pytest.mark.parametrize("variant", [S, NS])
@pytest.mark.parametrize("causal", [False, True])
def test_dV_is_attention_transpose(variant, causal):
    """C10: O is linear in V, O = A V with A the normalised (masked) kernel
    matrix, so dV = A^T dO."""
    Q, K, V, W1, W2, tau = _small_inputs(variant, seed=12)
    dO = _rng(13).standard_normal(V.shape)
    g = orc.linattn_bwd(Q, K, V, W1, W2, tau, dO, variant, causal)
    _, den, A = _quadratic(Q, K, V, W1, W2, tau, variant, causal)
    An = A / den[..., None]
    np.testing.assert_allclose(g["dV"], np.matmul(np.swapaxes(An, -1, -2), dO),
                               rtol=1e-9, atol=1e-10)


def _loss(Q, K, V, W1, W2, tau, dO, variant, causal):
    O, _ = orc.linattn_fwd(Q, K, V, W1, W2, tau, variant, causal)
    return float(np.sum(O * dO))


@pytest.mark.parametrize("variant", [S, NS])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("dv", [None, 5])
def test_finite_differences(variant, causal, dv):
    """C8: every analytic gradient (dQ, dK, dV, dW1, dW2, dtau) matches central
    finite differences of L = sum(O * dO), also with a value width other than d."""
    Q, K, V, W1, W2, tau = _small_inputs(variant, seed=14, B=1, H=2, N=6, d=3, m=4, scale=0.5, dv=dv)
    dO = _rng(15).standard_normal(V.shape)
    g = orc.linattn_bwd(Q, K, V, W1, W2, tau, dO, variant, causal, return_aux=True)
    # the query-side norm-factor gradient vanishes identically
    assert np.max(np.abs(g["g_q"])) < 1e-10 * max(1.0, np.max(np.abs(g["g_k"])))
    args = dict(Q=Q, K=K, V=V, W1=W1, W2=W2, tau=tau.astype(np.float64))
    names = ["Q", "K", "V", "W1", "tau"] + (["W2"] if variant == NS else [])
    h = 1e-6
    for name in names:
        base = args[name]
        fd = np.zeros_like(base)
        it = np.nditer(base, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            plus = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in args.items()}
            minus = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in args.items()}
            plus[name][idx] += h
            minus[name][idx] -= h
            fd[idx] = (_loss(dO=dO, variant=variant, causal=causal, **plus)
                       - _loss(dO=dO, variant=variant, causal=causal, **minus)) / (2 * h)
        an = g["d" + name]
        rel = np.linalg.norm(an - fd) / np.linalg.norm(fd)
        assert rel < 1e-6, (name, rel)


# --- attention-weight distillation loss L_awd (App. A.3, used in Sec. 4.3) ----

def _awd_inputs(variant, seed, B=2, H=2, N=7, d=4, m=5, scale=0.4, wscale=0.5):
    r = _rng(seed)
    W1 = r.standard_normal((H, m, d)) * wscale
    W2 = r.standard_normal((H, m, d)) * wscale if variant == NS else None
    Q = r.standard_normal((B, H, N, d)) * scale
    K = r.standard_normal((B, H, N, d)) * scale
    tau = np.array([math.log(2.0), 0.7])[:H]
    return Q, K, W1, W2, tau


def _entropy_rows(Q, K):
    """Mean row entropy of the softmax target, from scipy's softmax."""
    from scipy.special import softmax
    P = softmax(np.matmul(Q, np.swapaxes(K, -1, -2)) / math.sqrt(Q.shape[-1]), axis=-1)
    return -(P * np.log(P)).sum(-1).mean(-1), P


@pytest.mark.parametrize("variant", [S, NS])
def test_awd_zero_frequencies_closed_form(variant):
    """W = 0: every cosine is 1 and every sine 0, so A_ij = s^2 m e(Q_i) e(K_j)
    and the kernel's normalised weights are softmax_j(||K_j||^2 / c) for every
    query.  Then L = -(1/N) sum_ij P_ij ||K_j||^2 / c + logsumexp_l ||K_l||^2 / c,
    and with keys of equal norm L = log N exactly."""
    from scipy.special import logsumexp
    Q, K, W1, W2, tau = _awd_inputs(variant, seed=31)
    W1 = np.zeros_like(W1)
    W2 = None if W2 is None else np.zeros_like(W2)
    c = np.exp(tau)[None, :, None]
    u = (K * K).sum(-1) / c
    _, P = _entropy_rows(Q, K)
    expected = -(P * u[..., None, :]).sum(-1).mean(-1) + logsumexp(u, axis=-1)
    L = orc.awd_loss(Q, K, W1, W2, tau, variant)
    assert np.allclose(L, expected, rtol=1e-12, atol=1e-12)
    Ke = K / np.linalg.norm(K, axis=-1, keepdims=True) * 0.7
    L = orc.awd_loss(Q, Ke, W1, W2, tau, variant)
    assert np.allclose(L, math.log(Q.shape[-2]), rtol=0, atol=1e-12)


def test_awd_large_m_reaches_softmax_entropy():
    """Gaussian frequencies of variance 1/sqrt(d) with c = 2 sqrt(d) make
    phi~(x)^T phi~(y) an unbiased estimate of exp(x^T y / sqrt(d)) (the RFA form
    of the softmax kernel, Sec. 3.1); as m grows the kernel's weights approach
    the softmax target and L_awd approaches its lower bound, the mean row
    entropy of the target (Gibbs' inequality).  L >= entropy at every m."""
    r = _rng(33)
    B, H, N, d = 1, 1, 8, 4
    Q = r.standard_normal((B, H, N, d)) * 0.8
    K = r.standard_normal((B, H, N, d)) * 0.8
    tau = np.array([math.log(2.0 * math.sqrt(d))])
    Hm, _ = _entropy_rows(Q, K)
    gaps = []
    for m in (16, 2 ** 16):
        W = r.standard_normal((H, m, d)) * d ** -0.25
        L = orc.awd_loss(Q, K, W, None, tau, S)
        assert np.all(L >= Hm - 1e-12)
        gaps.append(float((L - Hm).max()))
    assert gaps[1] < 2e-3 < gaps[0]


@pytest.mark.parametrize("variant", [S, NS])
def test_awd_invariances(variant):
    """Permuting the keys (with their softmax logits) leaves every row's sum
    over j unchanged; sigma scales every A_ij alike and cancels in A_ij / den_i;
    Gibbs' inequality bounds L below by the target's mean row entropy."""
    Q, K, W1, W2, tau = _awd_inputs(variant, seed=35, m=32, wscale=0.4)
    L = orc.awd_loss(Q, K, W1, W2, tau, variant)
    assert np.all(np.isfinite(L))
    perm = _rng(36).permutation(K.shape[-2])
    assert np.allclose(orc.awd_loss(Q, K[..., perm, :], W1, W2, tau, variant), L, rtol=1e-12, atol=0)
    assert np.allclose(orc.awd_loss(Q, K, W1, W2, tau, variant, sigma=2.5), L, rtol=1e-12, atol=0)
    Hm, _ = _entropy_rows(Q, K)
    assert np.all(L >= Hm - 1e-12)


@pytest.mark.parametrize("variant", [S, NS])
def test_awd_query_norm_gradient_vanishes(variant):
    """L_awd depends on A_ij / sum_l A_il only, which no rescaling of phi(Q_i)
    changes: <phi(Q_i), dL/dphi(Q_i)> = 0 for every query, so the query norm
    factor contributes nothing to dtau (the key side does)."""
    Q, K, W1, W2, tau = _awd_inputs(variant, seed=39, m=32, wscale=0.4)
    g = orc.awd_grads(Q, K, W1, W2, tau, variant)
    pq = orc.feature_map(Q, W1, W2, tau, variant)
    pk = orc.feature_map(K, W1, W2, tau, variant)
    gq = (pq * g["dphi_q"]).sum(-1)
    gk = (pk * g["dphi_k"]).sum(-1)
    scale = np.abs(pq * g["dphi_q"]).sum(-1).max()
    assert np.abs(gq).max() <= 1e-12 * scale
    assert np.abs(gk).max() > 1e-3 * np.abs(pk * g["dphi_k"]).sum(-1).max()


def test_awd_nonpositive_ratio_gives_nan():
    """The log is taken as printed: one frequency at pi between a query and a
    key makes a kernel weight negative, and that slice's loss is NaN."""
    W = np.array([[[1.0]]])
    Q = np.zeros((1, 1, 2, 1))
    K = np.array([[[[0.0], [math.pi]]]])
    L = orc.awd_loss(Q, K, W, None, np.array([3.0]), S)
    assert np.isnan(L).all()


@pytest.mark.parametrize("variant", [S, NS])
def test_awd_finite_differences(variant):
    """dW1, dW2 and dtau of sum_{b,h} L_awd match central finite differences."""
    Q, K, W1, W2, tau = _awd_inputs(variant, seed=37, B=2, H=2, N=5, d=3, m=4, scale=0.4, wscale=0.6)
    g = orc.awd_grads(Q, K, W1, W2, tau, variant)
    assert np.all(np.isfinite(g["loss"]))
    args = dict(W1=W1, W2=W2, tau=tau.astype(np.float64))
    names = ["W1", "tau"] + (["W2"] if variant == NS else [])

    def total(**kw):
        return float(orc.awd_loss(Q, K, kw["W1"], kw["W2"], kw["tau"], variant).sum())

    h = 1e-6
    for name in names:
        base = args[name]
        fd = np.zeros_like(base)
        it = np.nditer(base, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            plus = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in args.items()}
            minus = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in args.items()}
            plus[name][idx] += h
            minus[name][idx] -= h
            fd[idx] = (total(**plus) - total(**minus)) / (2 * h)
        an = g["d" + name]
        rel = np.linalg.norm(an - fd) / np.linalg.norm(fd)
        assert rel < 1e-6, (name, rel)
