"""Plain float64 CPU oracle of GRKV's key step (the local linearized dual ridge
update of the retained keys).

TEST INFRASTRUCTURE ONLY, like ``grkv_oracle``: imported by the test suite,
the smoke check and the benchmark's CPU-baseline leg, never by the product
path, and sharing no code with the HIP path.

The key step (Sec. 3.4 "Key step" and "Linearized dual solution", Eq. 9-10;
Algorithm 1, key step; App. D.2 "Local Dual Key Update"; App. D.3 for fixed
tokens), with the values V fixed at the value step's result:

* f(K) = softmax(Q K^T / sqrt(d)) V over the retained keys (same causal rule as
  everywhere else), E = Y - f(K_cur), G = K_cur - K0 (zero at S = 1, where
  K_cur = K0), and J_G the derivative of f with respect to the free keys;
* alpha = (J_G J_G^T + lambda_k I_md)^-1 (vec(E) + J_G vec(G_G));
* K*_G = K0_G + unvec(J_G^T alpha), K*_F = K0_F.

J_G is never formed here either (App. D.2 applies J and J^T matrix-free): J_G[dK]
is the chain rule through the softmax and J_G^T alpha is its adjoint, both
written out below.  The dual system is solved to convergence (conjugate
gradients in float64 to a relative residual of 1e-12, or a dense solve on tiny
problems), i.e. the oracle computes the exact minimiser of the linearized
problem; how far a solver stops short of it is the solver's own tolerance.
The primal form (normal equations over the cd free key entries, App. D.2) is
provided for tiny problems as a cross-check of the dual identity.

``grkv_alternating`` runs Algorithm 1 with S > 1 alternating steps: at step t
the value step is taken at the current keys K^(t) (X from K^(t), the residual
anchored at V0), then the key step linearizes at K^(t) with the new values
(G = K^(t) - K0 no longer zero), and the loop stops after S steps or once the
largest change of K and V is at most 1e-9.

Parity status: pinned by ``tests/test_oracle_key.py`` (central finite
differences of f for J, adjointness of J and J^T, the primal = dual identity
against an explicit Jacobian, KKT conditions, limits in lambda_k, and a scalar
closed form).
"""
from __future__ import annotations

import math

import numpy as np

from . import grkv_oracle as V

__all__ = [
    "attention_output", "key_jvp", "key_vjp", "key_operator", "conjugate_gradient",
    "key_step", "key_primal", "grkv_unit", "grkv_alternating",
]


def attention_output(Q, K, Vr, idx, pos, causal):
    """f(K) = softmax(Q K^T / sqrt(d)) V over the retained keys K (positions
    idx), with the window rows' causal rule; returns (f, X)."""
    X = V.retained_attention(Q, K, idx, pos, causal)
    return X @ Vr, X


def key_jvp(Q, X, Vr, dK, free):
    """J_G[dK]: the first-order change of f when the free keys move by dK
    (rows of fixed tokens are ignored).  The logits change by
    dL = Q dK^T / sqrt(d); a row softmax changes by dX = X o (dL - rowsum(X o dL));
    the output by dX V."""
    d = Q.shape[1]
    dKg = np.where(free[:, None], dK, 0.0)
    dL = (Q @ dKg.T) / math.sqrt(d)
    dX = X * (dL - np.sum(X * dL, axis=1, keepdims=True))
    return dX @ Vr


def key_vjp(Q, X, Vr, alpha, free):
    """J_G^T alpha: the gradient of <alpha, f(K)> with respect to the free keys
    (zero rows for fixed tokens).  By the chain rule, gX = alpha V^T,
    gL = X o (gX - rowsum(X o gX)), gK = gL^T Q / sqrt(d)."""
    d = Q.shape[1]
    gX = alpha @ Vr.T
    gL = X * (gX - np.sum(X * gX, axis=1, keepdims=True))
    gK = (gL.T @ Q) / math.sqrt(d)
    gK[~free] = 0.0
    return gK


def key_operator(Q, X, Vr, free, lam_k):
    """alpha -> (J_G J_G^T + lambda_k I) alpha on [m, d] matrices."""
    def apply(a):
        return key_jvp(Q, X, Vr, key_vjp(Q, X, Vr, a, free), free) + lam_k * a
    return apply


def conjugate_gradient(apply, b, tol=1e-12, max_iter=None):
    """Conjugate gradients for a symmetric positive definite operator, started
    at zero (App. D.2 solves the dual system this way).  Stops when
    ||b - A x|| <= tol ||b|| (recursively updated residual).  Returns
    (x, iterations, final relative residual)."""
    x = np.zeros_like(b)
    r = b.copy()
    p = r.copy()
    rr = float(np.sum(r * r))
    bb = rr
    if bb == 0.0:
        return x, 0, 0.0
    max_iter = max_iter or b.size
    it = 0
    while it < max_iter and math.sqrt(rr) > tol * math.sqrt(bb):
        Ap = apply(p)
        a = rr / float(np.sum(p * Ap))
        x = x + a * p
        r = r - a * Ap
        rr_new = float(np.sum(r * r))
        p = r + (rr_new / rr) * p
        rr = rr_new
        it += 1
    return x, it, math.sqrt(rr / bb)


def key_step(Q, K0, Kcur, Vr, Y, idx, pos, fixed, lam_k, causal=True,
             solver="cg", tol=1e-12, max_iter=None):
    """One key step (Algorithm 1, key step; Eq. 9-10; App. D.2-D.3).

    Q [m, d] stacked window rows, K0 [c, d] the retained keys after eviction,
    Kcur [c, d] the current keys (K0 at S = 1), Vr [c, d] the values after the
    value step, Y [m, d] the full-cache target, idx [c] retained positions,
    pos [m] row positions, fixed [c] bool.  ``solver`` is "cg" (float64
    conjugate gradients) or "dense" (the md x md dual matrix built by applying
    the operator to unit vectors; tiny problems only).
    Returns a dict with E, the right-hand side rK, alpha, K* and solver info."""
    free = ~np.asarray(fixed, dtype=bool)
    fK, X = attention_output(Q, Kcur, Vr, idx, pos, causal)
    E = Y - fK
    Gd = np.where(free[:, None], Kcur - K0, 0.0)
    rK = E + key_jvp(Q, X, Vr, Gd, free)
    apply = key_operator(Q, X, Vr, free, lam_k)
    if solver == "dense":
        m, d = rK.shape
        M = np.empty((m * d, m * d))
        for col in range(m * d):
            e = np.zeros(m * d)
            e[col] = 1.0
            M[:, col] = apply(e.reshape(m, d)).ravel()
        alpha = np.linalg.solve(M, rK.ravel()).reshape(m, d)
        it, rel = m * d, float(np.linalg.norm(apply(alpha) - rK) / max(np.linalg.norm(rK), 1e-300))
    else:
        alpha, it, rel = conjugate_gradient(apply, rK, tol=tol, max_iter=max_iter)
    dK = key_vjp(Q, X, Vr, alpha, free)
    Kstar = K0 + dK
    return dict(E=E, rK=rK, X=X, fK=fK, alpha=alpha, dK=dK, Kstar=Kstar,
                iterations=it, rel_residual=rel)


def key_primal(Q, K0, Kcur, Vr, Y, idx, pos, fixed, lam_k, causal=True):
    """Primal form of the local ridge problem (App. D.2) on tiny problems:
    with the explicit Jacobian J_G (md x cd, one column per free key entry),
    solve (J^T J + lambda_k I) z = J^T (e + J g) over the free entries and
    return K* = K0 + unvec(z)."""
    free = ~np.asarray(fixed, dtype=bool)
    c, d = K0.shape
    fK, X = attention_output(Q, Kcur, Vr, idx, pos, causal)
    e = (Y - fK).ravel()
    cols, keys = [], []
    for j in np.flatnonzero(free):
        for dd in range(d):
            dK = np.zeros((c, d))
            dK[j, dd] = 1.0
            cols.append(key_jvp(Q, X, Vr, dK, free).ravel())
            keys.append((j, dd))
    Kstar = K0.copy()
    if not cols:
        return Kstar
    J = np.stack(cols, axis=1)
    g = np.array([(Kcur - K0)[j, dd] for j, dd in keys])
    z = np.linalg.solve(J.T @ J + lam_k * np.eye(J.shape[1]), J.T @ (e + J @ g))
    for (j, dd), v in zip(keys, z):
        Kstar[j, dd] = K0[j, dd] + v
    return Kstar


def grkv_unit(q_obs, K, Vfull, window, budget, pool_kernel, lam_v, lam_k, opt=None,
              idx=None, solver="cg", tol=1e-12):
    """Algorithm 1 with one alternating step (S = 1, the paper's default):
    selection and the value step (``grkv_oracle.compress_unit``), then the key
    step at K_cur = K0 with the merged values.  Returns the value-step dict
    with ``Kstar`` and the key-step dict under ``key``."""
    opt = opt or V.Options()
    r = V.compress_unit(q_obs, K, Vfull, window, budget, pool_kernel, lam_v, opt, idx=idx)
    ks = key_step(r["Q"], r["K0"], r["K0"], r["Vstar"], r["Y"], r["idx"], r["pos"],
                  r["fixed"], lam_k, opt.causal_window, solver=solver, tol=tol)
    r["key"] = ks
    r["Kstar"] = ks["Kstar"]
    return r


def grkv_alternating(q_obs, K, Vfull, window, budget, pool_kernel, lam_v, lam_k, steps, opt=None,
                     idx=None, tol=1e-12, stop=1e-9):
    """Algorithm 1 with up to ``steps`` alternating value/key steps.

    Step t (from K^(0) = K0, V^(0) = V0): X = softmax(Q K^(t)^T / sqrt(d)) over
    the retained keys; R_V = Y - X V0 (the value update stays anchored at V0);
    V^(t+1)_G = V0_G + X_G^T (X_G X_G^T + lambda_v I)^-1 R_V; then the key step
    at K_cur = K^(t) with V^(t+1) gives K^(t+1).  Stops early when
    max(max|K^(t+1) - K^(t)|, max|V^(t+1) - V^(t)|) <= stop.  Returns the
    value-step dict of the first step with ``Kstar``/``Vstar`` replaced by the
    final iterates, plus ``steps_run`` and per-step ``history``."""
    opt = opt or V.Options()
    r = V.compress_unit(q_obs, K, Vfull, window, budget, pool_kernel, lam_v, opt, idx=idx)
    Q, pos, ridx, F, Y = r["Q"], r["pos"], r["idx"], r["fixed"], r["Y"]
    K0, V0 = r["K0"], r["V0"]
    causal = opt.causal_window
    Kt, Vt = K0.copy(), V0.copy()
    history = []
    t = 0
    for t in range(steps):
        X = V.retained_attention(Q, Kt, ridx, pos, causal)
        dV, Z, R, status = V.merge_dual(X, Y, V0, F, lam_v)
        Vn = V0 + dV
        ks = key_step(Q, K0, Kt, Vn, Y, ridx, pos, F, lam_k, causal, tol=tol)
        Kn = ks["Kstar"]
        dk = float(np.abs(Kn - Kt).max()) if Kn.size else 0.0
        dv = float(np.abs(Vn - Vt).max()) if Vn.size else 0.0
        history.append(dict(X=X, Z=Z, Vstar=Vn, Kstar=Kn, key=ks, delta_k=dk, delta_v=dv,
                            status=status))
        Kt, Vt = Kn, Vn
        if max(dk, dv) <= stop:
            break
    out = dict(r)
    out.update(Kstar=Kt, Vstar=Vt, steps_run=t + 1, history=history)
    return out
