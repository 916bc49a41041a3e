"""Float64 CPU oracle for Flexformer's random-Fourier-feature linear attention.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the test suite, the smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code with the HIP path.

Plain, slow, float64 NumPy.  Every function follows a passage of the paper
(Flexformer, arXiv 2606.27748) and is cited by section / equation:

* feature maps      -- Sec. 3.1 Eq.(phi_n) with the norm factor of Eq.(softmax
                       kernel); Sec. 3.2 Eq.(phi_non) with the learnable norm
                       scale exp(tau) (paragraph "Flexformer with learnable
                       nonstationary kernel").
* attention         -- Sec. 2.2 Eq.(linear att), the state form
                       S = sum_j phi(K_j) V_j^T, z = sum_j phi(K_j).
* causal attention  -- the same state form restricted to j <= i (the paper's
                       autoregressive language model, Sec. 4.2, uses it; the
                       formula is not printed, so the mask is read as
                       inclusive).  Evaluated token by token as a running state.
* backward          -- derived by hand from the two forms above (the paper has
                       no backward); pinned by finite differences in the tests.
* decode step       -- the causal state form taken one token at a time (the
                       autoregressive language model of Sec. 4.2); pinned by
                       brute-force quadratic attention over the prefix.
* distillation loss -- the attention-weight distillation loss L_awd of
                       App. A.3 (used in Sec. 4.3): cross-entropy between the
                       softmax attention weights and the kernel's normalised
                       weights, and its gradient with respect to the kernel
                       parameters W1, W2, tau (derived here; pinned by a closed
                       form at W = 0, softmax recovery at large m, invariances
                       and finite differences).

Readings of the paper taken here:
  * nonstationary scale s = sigma / (2 sqrt(m)) as printed (its derivation
    drops a factor 4; the constant cancels in O and every gradient);
  * both variants use the norm factor exp(||x||^2 / exp(tau)) with a per-head
    tau; the frequencies are per head;
  * features are ordered [cos block | sin block] as printed;
  * no clamp or epsilon on the denominator;
  * L_awd: the log of A_ij / sum_l A_il is taken as printed (a non-positive
    ratio gives NaN or inf for its slice); the softmax target is a constant
    (only the kernel parameters are trained in the paper's distillation), and
    its logits are Q_i^T K_j / sqrt(d) as printed.

Every function here is pinned by a test in tests/test_oracle_pins.py; none is
"parity unpinned".
"""
from __future__ import annotations

import numpy as np

STATIONARY = "stationary"
NONSTATIONARY = "nonstationary"


# ----------------------------------------------------------------------------
# Frequencies and feature map
# ----------------------------------------------------------------------------

def nonstationary_pairs(W1, W2):
    """omega'_1 = (omega_1 + omega_2)/2, omega'_2 = (omega_1 - omega_2)/2
    (Sec. 3.2, definitions following Eq.(phi_non))."""
    W1 = np.asarray(W1, np.float64)
    W2 = np.asarray(W2, np.float64)
    return (W1 + W2) / 2.0, (W1 - W2) / 2.0


def _project(X, W):
    """P[b,h,n,k] = omega_k^T x_n for per-head frequencies W [H,m,d]."""
    return np.matmul(X, np.swapaxes(np.asarray(W, np.float64), -1, -2)[None])


def norm_factor(X, tau):
    """exp(||x||^2 / exp(tau)) per row (Sec. 3.2: the blue term of
    Eq.(softmax kernel) with 2 sqrt(d) replaced by exp(tau)); tau is per head."""
    c = np.exp(np.asarray(tau, np.float64))[None, :, None]
    with np.errstate(over="ignore"):
        return np.exp(np.sum(X * X, axis=-1) / c)


def feature_map_parts(X, W1, W2, tau, variant, sigma=1.0):
    """Feature map with its intermediates (used again by the backward).

    Stationary (Eq.(phi_n)): phi(x) = s e(x) [cos(Wx) ; sin(Wx)], s = sigma/sqrt(m).
    Nonstationary (Eq.(phi_non)): phi(x) = s e(x) [cos(W'1 x) cos(W'2 x) ;
    sin(W'1 x) cos(W'2 x)], s = sigma/(2 sqrt(m)).
    """
    X = np.asarray(X, np.float64)
    m = np.asarray(W1).shape[-2]
    e = norm_factor(X, tau)[..., None]
    if variant == STATIONARY:
        s = sigma / np.sqrt(m)
        P = _project(X, W1)
        phi = s * e * np.concatenate([np.cos(P), np.sin(P)], axis=-1)
        return phi, dict(s=s, e=e, P=P)
    if variant == NONSTATIONARY:
        s = sigma / (2.0 * np.sqrt(m))
        W1p, W2p = nonstationary_pairs(W1, W2)
        P1 = _project(X, W1p)
        P2 = _project(X, W2p)
        phi = s * e * np.concatenate([np.cos(P1) * np.cos(P2),
                                      np.sin(P1) * np.cos(P2)], axis=-1)
        return phi, dict(s=s, e=e, P1=P1, P2=P2, W1p=W1p, W2p=W2p)
    raise ValueError(variant)


def feature_map(X, W1, W2, tau, variant, sigma=1.0):
    """phi~(x) for X [B,H,N,d] -> [B,H,N,2m] (Sec. 3.1/3.2)."""
    return feature_map_parts(X, W1, W2, tau, variant, sigma)[0]


# ----------------------------------------------------------------------------
# Attention forward (Eq.(linear att))
# ----------------------------------------------------------------------------

def _augment(V):
    """[V | 1]: the value rows with the normaliser column appended, so that one
    state holds S = sum phi(K) V^T and z = sum phi(K) (Eq.(linear att))."""
    V = np.asarray(V, np.float64)
    return np.concatenate([V, np.ones(V.shape[:-1] + (1,))], axis=-1)


def attend_features(phi_q, phi_k, V, causal):
    """[num | den] from feature rows, Eq.(linear att).

    Non-causal: S' = Phi_K^T [V|1]; [num|den]_i = phi(Q_i)^T S'.
    Causal: the running state S'_i = sum_{j<=i} phi(K_j)[V_j;1]^T is updated
    token by token and read out by phi(Q_i).
    Returns (num [B,H,N,dv], den [B,H,N]).
    """
    Vp = _augment(V)
    if not causal:
        S = np.matmul(np.swapaxes(phi_k, -1, -2), Vp)
        nd = np.matmul(phi_q, S)
    else:
        B, H, N, Dp = phi_q.shape
        S = np.zeros((B, H, Dp, Vp.shape[-1]))
        nd = np.empty(phi_q.shape[:-1] + (Vp.shape[-1],))
        for i in range(N):
            S += phi_k[:, :, i, :, None] * Vp[:, :, i, None, :]
            nd[:, :, i, :] = np.einsum("bhf,bhfv->bhv", phi_q[:, :, i, :], S)
    return nd[..., :-1], nd[..., -1]


def decode_step(state, q, k, v, W1, W2, tau, variant, sigma=1.0):
    """One step of causal attention as a recurrence (the autoregressive use of
    Eq.(linear att) in Sec. 4.2): the state S' = sum_j phi(k_j) [v_j ; 1]^T
    takes the new token, then the new query reads it out (inclusive mask).

    state [B,H,2m,dv+1] (feature rows in [cos | sin] order, last column the
    normaliser z); q, k [B,H,d]; v [B,H,dv].  Returns (o [B,H,dv], den [B,H],
    new state); the input state is not modified.
    """
    q = np.asarray(q, np.float64)[:, :, None, :]
    k = np.asarray(k, np.float64)[:, :, None, :]
    phi_q = feature_map(q, W1, W2, tau, variant, sigma)[:, :, 0, :]
    phi_k = feature_map(k, W1, W2, tau, variant, sigma)[:, :, 0, :]
    vp = np.concatenate([np.asarray(v, np.float64), np.ones(np.shape(v)[:-1] + (1,))], axis=-1)
    S = np.asarray(state, np.float64) + phi_k[..., :, None] * vp[..., None, :]
    nd = np.einsum("bhf,bhfv->bhv", phi_q, S)
    return nd[..., :-1] / nd[..., -1:], nd[..., -1], S


def linattn_fwd(Q, K, V, W1, W2, tau, variant, causal, sigma=1.0):
    """O = num / den (Eq.(linear att)), no clamp on den.  Returns (O, den)."""
    pq = feature_map(Q, W1, W2, tau, variant, sigma)
    pk = feature_map(K, W1, W2, tau, variant, sigma)
    num, den = attend_features(pq, pk, V, causal)
    with np.errstate(divide="ignore", invalid="ignore"):
        O = num / den[..., None]
    return O, den


def linattn_fwd_rows(Q, K, V, W1, W2, tau, variant, causal, rows, sigma=1.0):
    """O and den for selected (b, h, i) rows only, each from its own sums
    sum_{j} phi(Q_i)^T phi(K_j) [V_j;1] over j <= i (causal) or all j.
    ``rows`` is an int array [R,3] of (b, h, i).  For full-size spot checks."""
    rows = np.asarray(rows)
    out_O = np.empty((len(rows), np.asarray(V).shape[-1]))
    out_den = np.empty(len(rows))
    for r, (b, h, i) in enumerate(rows):
        sl = slice(None, i + 1) if causal else slice(None)
        q = np.asarray(Q, np.float64)[b:b + 1, h:h + 1, i:i + 1]
        k = np.asarray(K, np.float64)[b:b + 1, h:h + 1, sl]
        v = np.asarray(V, np.float64)[b:b + 1, h:h + 1, sl]
        Wa = np.asarray(W1)[h:h + 1]
        Wb = None if W2 is None else np.asarray(W2)[h:h + 1]
        t = np.asarray(tau)[h:h + 1]
        pq = feature_map(q, Wa, Wb, t, variant, sigma)
        pk = feature_map(k, Wa, Wb, t, variant, sigma)
        nd = np.matmul(np.matmul(pq, np.swapaxes(pk, -1, -2)), _augment(v))[0, 0, 0]
        out_den[r] = nd[-1]
        with np.errstate(divide="ignore", invalid="ignore"):
            out_O[r] = nd[:-1] / nd[-1]
    return out_O, out_den


def conditioning(Q, K, W1, W2, tau, variant, causal, sigma=1.0, return_den=False):
    """kappa_i = sum_k |phi(Q_i)_k z_ik| / |den_i|, z_i = sum_{j(<=i)} phi(K_j):
    the condition number of the denominator's dot product.  With trigonometric
    features den is sign-indefinite, and a row's rounding error grows with
    kappa_i; parity tests weight rows by it.  With return_den, also the
    den_i = sum_k phi(Q_i)_k z_ik the condition numbers belong to."""
    pq = feature_map(Q, W1, W2, tau, variant, sigma)
    pk = feature_map(K, W1, W2, tau, variant, sigma)
    z = np.cumsum(pk, axis=-2) if causal else np.broadcast_to(
        pk.sum(axis=-2, keepdims=True), pk.shape)
    t = pq * z
    den = t.sum(-1)
    with np.errstate(divide="ignore", invalid="ignore"):
        kappa = np.abs(t).sum(-1) / np.abs(den)
    return (kappa, den) if return_den else kappa


# ----------------------------------------------------------------------------
# Backward
# ----------------------------------------------------------------------------

def _feature_map_bwd(X, parts, phi, dphi, variant, tau):
    """Chain rule through phi~ for one input X.

    Returns (dX, dW1, dW2, dtau) with dW* summed over batch and rows.
    Stationary: dP = -Phi_sin * dPhi_cos + Phi_cos * dPhi_sin; dX = dP W.
    Nonstationary: with Phi_a = s e cos P1 cos P2, Phi_b = s e sin P1 cos P2,
      dP1 = -Phi_b dPhi_a + Phi_a dPhi_b,
      dP2 = -s e sin P2 (cos P1 dPhi_a + sin P1 dPhi_b),
      dX = dP1 W'1 + dP2 W'2, and (dW1, dW2) = ((dW'1 + dW'2)/2, (dW'1 - dW'2)/2)
      because W'1 = (W1 + W2)/2 and W'2 = (W1 - W2)/2.
    Norm factor e = exp(||x||^2 / c), c = exp(tau): with g = <phi, dphi>,
      dX += (2/c) g x and dtau = -sum g ||x||^2 / c.
    """
    X = np.asarray(X, np.float64)
    m = phi.shape[-1] // 2
    c = np.exp(np.asarray(tau, np.float64))[None, :, None]
    g = np.sum(phi * dphi, axis=-1)                      # [B,H,N]
    sq = np.sum(X * X, axis=-1)
    da, db = dphi[..., :m], dphi[..., m:]
    pa, pb = phi[..., :m], phi[..., m:]
    if variant == STATIONARY:
        dP = -pb * da + pa * db
        dX = np.matmul(dP, np.asarray(parts.get("W"), np.float64)[None])
        dW1 = np.matmul(np.swapaxes(dP, -1, -2), X).sum(axis=0)
        dW2 = None
    else:
        s, e, P1, P2 = parts["s"], parts["e"], parts["P1"], parts["P2"]
        dP1 = -pb * da + pa * db
        dP2 = -s * e * np.sin(P2) * (np.cos(P1) * da + np.sin(P1) * db)
        dX = (np.matmul(dP1, parts["W1p"][None]) + np.matmul(dP2, parts["W2p"][None]))
        dW1p = np.matmul(np.swapaxes(dP1, -1, -2), X).sum(axis=0)
        dW2p = np.matmul(np.swapaxes(dP2, -1, -2), X).sum(axis=0)
        dW1 = (dW1p + dW2p) / 2.0
        dW2 = (dW1p - dW2p) / 2.0
    dX = dX + (2.0 / c)[..., None] * g[..., None] * X
    dtau = -(g * sq / c).sum(axis=(0, 2))
    return dX, dW1, dW2, dtau, g


def linattn_bwd(Q, K, V, W1, W2, tau, dO, variant, causal, sigma=1.0, return_aux=False):
    """Gradients of the forward output O with respect to Q, K, V, W1, W2, tau
    for an upstream gradient dO (the paper has no backward; derivation):

      [num|den]_i = sum_j a_ij [V_j ; 1] with a_ij = phi(Q_i)^T phi(K_j) (j<=i if causal)
      G_i = [dO_i / den_i ; -(dO_i . O_i) / den_i]
      dphi(Q_i) = S'_i G_i,       S'_i = sum_{j(<=i)} phi(K_j) [V_j;1]^T
      dphi(K_j) = R'_j [V_j;1],   R'_j = sum_{i(>=j)} phi(Q_i) G_i^T
      dV_j      = (R'_j^T phi(K_j))[:dv]
    followed by the feature-map chain rule.  Returns a dict.
    """
    Q = np.asarray(Q, np.float64)
    K = np.asarray(K, np.float64)
    V = np.asarray(V, np.float64)
    dO = np.asarray(dO, np.float64)
    pq, parts_q = feature_map_parts(Q, W1, W2, tau, variant, sigma)
    pk, parts_k = feature_map_parts(K, W1, W2, tau, variant, sigma)
    num, den = attend_features(pq, pk, V, causal)
    with np.errstate(divide="ignore", invalid="ignore"):
        O = num / den[..., None]
        delta = np.sum(dO * O, axis=-1)
        G = np.concatenate([dO / den[..., None], (-delta / den)[..., None]], axis=-1)
    Vp = _augment(V)
    if not causal:
        S = np.matmul(np.swapaxes(pk, -1, -2), Vp)
        R = np.matmul(np.swapaxes(pq, -1, -2), G)
        dpq = np.matmul(G, np.swapaxes(S, -1, -2))
        dpk = np.matmul(Vp, np.swapaxes(R, -1, -2))
        dVp = np.matmul(pk, R)
    else:
        B, H, N, Dp = pq.shape
        Dv1 = Vp.shape[-1]
        dpq = np.empty_like(pq)
        dpk = np.empty_like(pk)
        dVp = np.empty((B, H, N, Dv1))
        S = np.zeros((B, H, Dp, Dv1))
        for i in range(N):
            S += pk[:, :, i, :, None] * Vp[:, :, i, None, :]
            dpq[:, :, i] = np.einsum("bhfv,bhv->bhf", S, G[:, :, i])
        R = np.zeros((B, H, Dp, Dv1))
        for j in range(N - 1, -1, -1):
            R += pq[:, :, j, :, None] * G[:, :, j, None, :]
            dpk[:, :, j] = np.einsum("bhfv,bhv->bhf", R, Vp[:, :, j])
            dVp[:, :, j] = np.einsum("bhfv,bhf->bhv", R, pk[:, :, j])
    dV = dVp[..., :-1]
    if variant == STATIONARY:
        parts_q["W"] = np.asarray(W1, np.float64)
        parts_k["W"] = np.asarray(W1, np.float64)
    dQ, dW1q, dW2q, dtq, gq = _feature_map_bwd(Q, parts_q, pq, dpq, variant, tau)
    dK, dW1k, dW2k, dtk, gk = _feature_map_bwd(K, parts_k, pk, dpk, variant, tau)
    out = dict(dQ=dQ, dK=dK, dV=dV, dW1=dW1q + dW1k,
               dW2=None if dW2q is None else dW2q + dW2k, dtau=dtq + dtk)
    if return_aux:
        out.update(O=O, den=den, g_q=gq, g_k=gk, G=G, phi_k=pk, dphi_k=dpk)
    return out


# ----------------------------------------------------------------------------
# Attention-weight distillation loss (App. A.3, used in Sec. 4.3)
# ----------------------------------------------------------------------------

def softmax_weights(Q, K):
    """P_ij = exp(Q_i^T K_j / sqrt(d)) / sum_l exp(Q_i^T K_l / sqrt(d)), the
    target attention weights of L_awd (row-wise softmax of the scaled logits)."""
    Q = np.asarray(Q, np.float64)
    K = np.asarray(K, np.float64)
    S = np.matmul(Q, np.swapaxes(K, -1, -2)) / np.sqrt(Q.shape[-1])
    S = S - S.max(axis=-1, keepdims=True)
    E = np.exp(S)
    return E / E.sum(axis=-1, keepdims=True)


def awd_loss(Q, K, W1, W2, tau, variant, sigma=1.0, return_aux=False):
    """L_awd of App. A.3 for every (b,h) slice:

      L = -(1/N) sum_i sum_j P_ij log( A_ij / sum_l A_il ),
      P = softmax_weights(Q, K),  A_ij = phi~(Q_i)^T phi~(K_j),

    phi~ being the variant's feature map with its norm factor.  Evaluated as
    printed (no clamp, no epsilon).  Returns L [B,H] (and the intermediates
    with return_aux)."""
    Q = np.asarray(Q, np.float64)
    K = np.asarray(K, np.float64)
    N = Q.shape[-2]
    pq, parts_q = feature_map_parts(Q, W1, W2, tau, variant, sigma)
    pk, parts_k = feature_map_parts(K, W1, W2, tau, variant, sigma)
    A = np.matmul(pq, np.swapaxes(pk, -1, -2))
    P = softmax_weights(Q, K)
    den = A.sum(axis=-1)
    with np.errstate(divide="ignore", invalid="ignore"):
        L = -(P * np.log(A / den[..., None])).sum(axis=-1).sum(axis=-1) / N
    if return_aux:
        return L, dict(A=A, P=P, den=den, pq=pq, pk=pk, parts_q=parts_q, parts_k=parts_k)
    return L


def awd_grads(Q, K, W1, W2, tau, variant, sigma=1.0):
    """Gradients of sum_{b,h} L_awd[b,h] with respect to W1, W2 and tau
    (derivation; the paper gives none).  With Sigma_j P_ij = 1,

      dL/dA_ij = G_ij = (1/N) (1/den_i - P_ij / A_ij),   den_i = sum_l A_il,
      dphi(Q_i) = sum_j G_ij phi(K_j),   dphi(K_j) = sum_i G_ij phi(Q_i),

    followed by the feature-map chain rule of the attention backward.
    Returns dict(loss, dW1, dW2, dtau, dphi_q, dphi_k)."""
    Q = np.asarray(Q, np.float64)
    K = np.asarray(K, np.float64)
    N = Q.shape[-2]
    L, aux = awd_loss(Q, K, W1, W2, tau, variant, sigma, return_aux=True)
    A, P, den, pq, pk = aux["A"], aux["P"], aux["den"], aux["pq"], aux["pk"]
    with np.errstate(divide="ignore", invalid="ignore"):
        G = (1.0 / den[..., None] - P / A) / N
    dpq = np.matmul(G, pk)
    dpk = np.matmul(np.swapaxes(G, -1, -2), pq)
    parts_q, parts_k = aux["parts_q"], aux["parts_k"]
    if variant == STATIONARY:
        parts_q["W"] = np.asarray(W1, np.float64)
        parts_k["W"] = np.asarray(W1, np.float64)
    _, dW1q, dW2q, dtq, _ = _feature_map_bwd(Q, parts_q, pq, dpq, variant, tau)
    _, dW1k, dW2k, dtk, _ = _feature_map_bwd(K, parts_k, pk, dpk, variant, tau)
    return dict(loss=L, dW1=dW1q + dW1k, dW2=None if dW2q is None else dW2q + dW2k,
                dtau=dtq + dtk, dphi_q=dpq, dphi_k=dpk)
