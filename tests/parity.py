"""Parity metrics between the HIP path and the float64 oracle.

The conditioning-aware reading of "relative error <= 1e-4 (fp32) / 2e-2
(bf16-input)": with trigonometric features the denominator
den_i = phi(Q_i).z_i is sign-indefinite, so a row's error grows with the
condition number kappa_i = sum_k |phi(Q_i)_k z_ik| / |den_i| of that dot
product, whatever the implementation.  Hence:

T1 (slices of at least 128 rows): per (b,h) slice, the Frobenius relative
    error of num = O * den (formed in float64) and of den, each <= tol.
T1a (every case): per (b,h) slice, the Frobenius norm of the num and den
    errors relative to the magnitude of the summed terms,
    num_abs = (|phi(Q)| |phi(K)|^T (.) mask) |V| and den_abs = the same with 1
    for |V|, <= tol.  Rounding the features to precision u perturbs num_i by at
    most ~u num_abs_i whatever the conditioning, so this holds for short
    sequences where every row may be ill-conditioned.
T2 (every case): over rows with kappa_i <= kappa_max, the Frobenius relative
    error of O <= tol; and every row i has rel_i <= max(tol, 4 u K_i), u the
    unit roundoff of the feature precision and K_i the condition number of
    O_i = num_i / den_i, den_abs_i/|den_i| + |num_abs_i|/|num_i| (kappa_i where
    the absolute scales are not computed).  A row whose den rounding bound
    4 u den_abs_i reaches |den_i| has no determined O_i at precision u; its
    num_i and den_i errors are bounded by 4 u num_abs_i and 4 u den_abs_i.
    A row whose den is exactly zero (O_i not finite; no epsilon is added) is
    checked on den_i alone, which passes only where den_i is not determined.
T3 (gradients): the upstream gradient is zeroed on rows with
    kappa_i > KAPPA_MAX_GRAD (identically for the oracle and the GPU); then the
    Frobenius relative error of every gradient <= tol.  dtau, a single sum
    over all key rows whose terms cancel, is measured relative to the
    magnitude of its summed terms (dtau_scale).
"""
from __future__ import annotations

import json
import os

import numpy as np


def _log(kind, stats):
    """Append the statistics of a check to $FLEX_PARITY_LOG (JSON lines), if set."""
    path = os.environ.get("FLEX_PARITY_LOG")
    if path:
        test = os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0]
        with open(path, "a") as f:
            f.write(json.dumps(dict(test=test, kind=kind, **stats)) + "\n")

TOL = {"f32": 1e-4, "bf16": 2e-2}
KAPPA_MAX = {"f32": 1e3, "bf16": 20.0}
# Gradients of a kept row depend on every other kept row (through the states),
# so their error is an average of c u kappa_i over kept rows; kappa_max is set
# so that u kappa_max stays well below the tolerance (fp32: 6e-8 * 1e3).
KAPPA_MAX_GRAD = {"f32": 1e3, "bf16": 20.0}
UNIT = {"f32": 2.0 ** -24, "bf16": 2.0 ** -9}


def frob_rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / nb) if nb > 0 else float(np.linalg.norm(a - b))


def abs_scales(x, wl):
    """(num_abs, den_abs) of T1a for seeded inputs x of workload wl (small N)."""
    import oracle as orc
    Q, K, V = x.f64("Q"), x.f64("K"), x.f64("V")
    pq = np.abs(orc.feature_map(Q, x.W1, x.W2, x.tau, wl.variant))
    pk = np.abs(orc.feature_map(K, x.W1, x.W2, x.tau, wl.variant))
    A = np.matmul(pq, np.swapaxes(pk, -1, -2))
    if wl.causal:
        A = np.tril(A)
    return np.matmul(A, np.abs(V)), A.sum(-1)


def check_forward(io, O_gpu, den_gpu, O_ref, den_ref, kappa, scales=None, rows_mask=None, t2_on=True):
    """Apply T1, T1a and T2; returns a dict of statistics and raises
    AssertionError with the statistics when a criterion fails.  t2_on=False
    leaves out T2's Frobenius bound (its statistic is still logged): for
    inputs where the precision alone reaches it."""
    tol, kmax, u = TOL[io], KAPPA_MAX[io], UNIT[io]
    O_gpu = np.asarray(O_gpu, np.float64)
    den_gpu = np.asarray(den_gpu, np.float64)
    num_ref = O_ref * den_ref[..., None]
    # A row whose den came out exactly zero has O_i = num_i / 0, not finite by
    # definition (no epsilon is added).  Its num_i cannot be recovered from O
    # and den, so it enters the num and O measures as exact and is checked on
    # den_i alone (below).
    zero = den_gpu == 0.0
    O_gpu = np.where(zero[..., None], O_ref, O_gpu)
    num_gpu = O_gpu * den_gpu[..., None]
    num_gpu = np.where(zero[..., None], num_ref, num_gpu)
    B, H, N = O_ref.shape[:3]
    t1n = max(frob_rel(num_gpu[b, h], num_ref[b, h]) for b in range(B) for h in range(H))
    t1d = max(frob_rel(den_gpu[b, h], den_ref[b, h]) for b in range(B) for h in range(H))
    t1an = t1ad = 0.0
    if scales is not None:
        num_abs, den_abs = scales
        t1an = max(float(np.linalg.norm(num_gpu[b, h] - num_ref[b, h]) / np.linalg.norm(num_abs[b, h]))
                   for b in range(B) for h in range(H))
        t1ad = max(float(np.linalg.norm(den_gpu[b, h] - den_ref[b, h]) / np.linalg.norm(den_abs[b, h]))
                   for b in range(B) for h in range(H))
    good = kappa <= kmax
    if rows_mask is not None:
        good &= rows_mask
    t2 = frob_rel(O_gpu[good], O_ref[good]) if good.any() else 0.0
    with np.errstate(divide="ignore", invalid="ignore"):
        rel = np.linalg.norm(O_gpu - O_ref, axis=-1) / np.linalg.norm(O_ref, axis=-1)
        if scales is not None:
            # condition number of O_i = num_i / den_i: that of den_i plus that of num_i
            num_abs, den_abs = scales
            kfull = den_abs / np.abs(den_ref) + (np.linalg.norm(num_abs, axis=-1)
                                                 / np.linalg.norm(num_ref, axis=-1))
        else:
            kfull = kappa
        bound = np.maximum(tol, 4 * u * kfull)
        ratio = rel / bound
        # absolute scale of den_i's rounding: the summed terms where they are
        # computed, else sum_k |phi(Q_i)_k z_ik| = kappa_i |den_i|
        den_scale = den_abs if scales is not None else kappa * np.abs(den_ref)
        r_den = np.abs(den_gpu - den_ref) / (4 * u * den_scale)
        if scales is not None:
            # O_i = num_i / den_i is first-order in the rounding only while the
            # rounding bound of den_i, 4 u den_abs_i, is below |den_i|.  Where
            # it is not, the sign of den_i is not fixed at this precision and
            # O_i can take any value: such rows are checked on num_i and den_i
            # against their absolute scales instead.
            undet = 4 * u * den_abs >= np.abs(den_ref)
            r_num = np.linalg.norm(num_gpu - num_ref, axis=-1) / (4 * u * np.linalg.norm(num_abs, axis=-1))
            ratio = np.where(undet, np.maximum(r_num, r_den), ratio)
        ratio = np.where(zero, r_den, ratio)
        worst = np.nanmax(ratio)
    stats = dict(T1_num=t1n, T1_den=t1d, T1a_num=t1an, T1a_den=t1ad, T2=t2, row_worst=float(worst),
                 rows_kept=float(good.mean()), den_le0=float((den_ref <= 0).mean()),
                 whole_O=frob_rel(O_gpu, O_ref), kappa_med=float(np.median(kappa)))
    ok = t1an <= tol and t1ad <= tol and (t2 <= tol or not t2_on) and worst <= 1.0
    if N >= 128:
        ok = ok and t1n <= tol and t1d <= tol
    _log("forward", stats)
    assert ok, stats
    return stats


def dtau_scale(x, wl, aux):
    """Magnitude of the summed terms of dtau = -sum_j <phi(K_j), dphi(K_j)> |k_j|^2 / c
    per head: sum_j sum_f |phi(K_j)_f dphi(K_j)_f| |k_j|^2 / c (oracle values)."""
    K = x.f64("K")
    c = np.exp(np.asarray(x.tau, np.float64))
    t = np.abs(aux["phi_k"] * aux["dphi_k"]).sum(-1) * (K * K).sum(-1) / c[None, :, None]
    return t.sum(axis=(0, 2))


ROW_TOL = {"f32": 5e-4, "bf16": 0.1}


def dv_row_scale(pq, pk, dO, den, kappa, causal):
    """Scale of the rounding error of each dV row (dV = A^T dO, Eq.(linear att)):
    s_j = sum_i sum_f |phi(Q_i)_f| |phi(K_j)_f| (1 + kappa_i) |dO_i| / |den_i|
    over i >= j (causal) or all i.  Rounding the features to precision u moves
    a_ij by at most ~u sum_f |phi_if phi_jf| and den_i by ~u kappa_i |den_i|,
    so |delta dV_j| <~ u s_j.  Formed as |phi(K_j)| . (suffix) sum_i w_i |phi(Q_i)|,
    O(N d') per slice.  Rows i whose dO is zero contribute nothing."""
    nrm = np.linalg.norm(dO, axis=-1)
    with np.errstate(divide="ignore", invalid="ignore"):
        w = np.where(nrm > 0, (1.0 + kappa) * nrm / np.abs(den), 0.0)
    t = w[..., None] * np.abs(pq)
    if causal:
        acc = np.flip(np.cumsum(np.flip(t, -2), axis=-2), -2)
    else:
        acc = np.broadcast_to(t.sum(-2, keepdims=True), t.shape)
    return (np.abs(pk) * acc).sum(-1)


def check_grad_rows(io, got: dict, ref: dict, names=("dQ", "dK", "dV"), dv_scale=None, n_terms=1):
    """Row-wise checks of [..., N, d] gradients, which a Frobenius norm over the
    whole tensor would not see for a single wrong row:

    * every row's error relative to max(|row|, RMS row norm) <= ROW_TOL
      (5 tol; a wrong row scores about 1).  Meant for slices of tens of rows
      or more: at N = 1, 2 the exact gradients of some rows vanish and every
      row may be rounding noise (those lengths have their own checks);
    * with dv_scale (dv_row_scale), |delta dV_j| <= (4 u + 4 u32 sqrt(n_terms)) s_j,
      u the feature precision and u32 the fp32 accumulation over n_terms rows."""
    stats = {}
    ok = True
    for n in names:
        g = np.asarray(got[n], np.float64)
        r = np.asarray(ref[n], np.float64)
        nr = np.linalg.norm(r, axis=-1)
        rms = float(np.sqrt(np.mean(nr * nr)))
        rr = np.linalg.norm(g - r, axis=-1) / np.maximum(nr, rms if rms > 0 else 1.0)
        stats[n + "_row_max"] = float(rr.max())
        ok = ok and stats[n + "_row_max"] <= ROW_TOL[io]
    if dv_scale is not None:
        e = np.linalg.norm(np.asarray(got["dV"], np.float64) - ref["dV"], axis=-1)
        bound = (4 * UNIT[io] + 4 * 2.0 ** -24 * np.sqrt(n_terms)) * dv_scale
        with np.errstate(divide="ignore", invalid="ignore"):
            q = np.where(bound > 0, e / bound, np.where(e > 0, np.inf, 0.0))
        stats["dV_row_bound"] = float(q.max())
        ok = ok and stats["dV_row_bound"] <= 1.0
    _log("grad_rows", stats)
    assert ok, stats
    return stats


def check_grads(io, got: dict, ref: dict, names, scales=None):
    """T3.  For names listed in `scales` the error is measured relative to the
    given magnitude of the summed terms instead of the value (dtau is a sum
    whose terms cancel)."""
    tol = TOL[io]
    scales = scales or {}
    stats = {}
    for n in names:
        if n in scales:
            stats[n] = float(np.linalg.norm(np.asarray(got[n], np.float64) - ref[n])
                             / np.linalg.norm(scales[n]))
            stats[n + "_plain"] = frob_rel(got[n], ref[n])
        else:
            stats[n] = frob_rel(got[n], ref[n])
    _log("grads", stats)
    assert all(stats[n] <= tol for n in names), stats
    return stats
