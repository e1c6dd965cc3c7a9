"""Pins for the oracle's key step (Sec. 3.4 key step, Eq. 9-10; Algorithm 1, key
step; App. D.2 local dual key update; App. D.3 fixed tokens).

The key step linearizes f(K) = softmax(Q K^T / sqrt(d)) V around the current
keys and solves the ridge problem min ||e - J d||^2 + lambda_k ||d + g||^2 in
its dual form.  Each test checks the oracle against something other than its
own formulas: finite differences of f itself, the adjoint identity, an
explicit Jacobian with the primal normal equations, a scalar closed form, the
optimality conditions and the limits of the problem.
"""
import math

import numpy as np
import pytest

import workloads as W
from oracle import grkv_key_oracle as KO
from oracle import grkv_oracle as O


def _problem(seed, m=6, c=9, d=4, n_fixed=2, causal=True, perturb=0.0, scale=1.0):
    """A small retained cache: positions idx (ascending, ending with the
    window), window rows at the last positions, random Q/K/V."""
    rng = np.random.default_rng(seed)
    w = 3
    n = 40
    G = m // w
    idx = np.sort(np.concatenate([rng.choice(n - w, c - w, replace=False), np.arange(n - w, n)]))
    pos = O.query_positions(G, w, n)
    Q = scale * rng.standard_normal((m, d))
    K0 = rng.standard_normal((c, d))
    Kcur = K0 + perturb * rng.standard_normal((c, d))
    Vr = rng.standard_normal((c, d))
    Y = rng.standard_normal((m, d))
    F = np.zeros(c, dtype=bool)
    F[rng.choice(c, n_fixed, replace=False)] = True
    return Q, K0, Kcur, Vr, Y, idx, pos, F, causal


def _f(Q, K, Vr, idx, pos, causal):
    # f written out independently: masked logits, max-shifted exponentials
    d = Q.shape[1]
    L = Q @ K.T / math.sqrt(d)
    if causal:
        L = np.where(idx[None, :] <= pos[:, None], L, -np.inf)
    e = np.exp(L - L.max(axis=1, keepdims=True))
    return (e / e.sum(axis=1, keepdims=True)) @ Vr


@pytest.mark.parametrize("causal", [True, False])
def test_jvp_matches_central_differences(causal):
    Q, K0, Kc, Vr, Y, idx, pos, F, _ = _problem(0, causal=causal)
    free = ~F
    _, X = KO.attention_output(Q, Kc, Vr, idx, pos, causal)
    rng = np.random.default_rng(1)
    for _ in range(5):
        dK = rng.standard_normal(Kc.shape)
        dKg = np.where(free[:, None], dK, 0.0)
        h = 1e-5
        fd = (_f(Q, Kc + h * dKg, Vr, idx, pos, causal) - _f(Q, Kc - h * dKg, Vr, idx, pos, causal)) / (2 * h)
        jv = KO.key_jvp(Q, X, Vr, dK, free)
        assert np.abs(jv - fd).max() <= 1e-8 * max(1.0, np.abs(fd).max())


def test_vjp_is_the_adjoint_of_jvp():
    Q, K0, Kc, Vr, Y, idx, pos, F, causal = _problem(2)
    free = ~F
    _, X = KO.attention_output(Q, Kc, Vr, idx, pos, causal)
    rng = np.random.default_rng(3)
    for _ in range(5):
        dK = rng.standard_normal(Kc.shape)
        a = rng.standard_normal(Y.shape)
        lhs = np.sum(a * KO.key_jvp(Q, X, Vr, dK, free))
        rhs = np.sum(KO.key_vjp(Q, X, Vr, a, free) * dK)
        assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))
    # fixed tokens: J^T alpha has zero rows, and J ignores their directions
    g = KO.key_vjp(Q, X, Vr, rng.standard_normal(Y.shape), free)
    assert np.all(g[F] == 0.0)
    dK = np.zeros_like(Kc)
    dK[F] = 1.0
    assert np.all(KO.key_jvp(Q, X, Vr, dK, free) == 0.0)


def test_scalar_closed_form():
    # one row, two keys, d = 1: f = p v1 + (1 - p) v2 with p = sigmoid(q (k1 - k2)),
    # so df/dk1 = q p (1 - p) (v1 - v2) and df/dk2 = -df/dk1
    q, k1, k2, v1, v2 = 0.7, 0.3, -1.1, 2.0, -0.5
    p = 1.0 / (1.0 + math.exp(-q * (k1 - k2)))
    d1 = q * p * (1 - p) * (v1 - v2)
    Q = np.array([[q]])
    K = np.array([[k1], [k2]])
    Vr = np.array([[v1], [v2]])
    idx = np.array([0, 1])
    pos = np.array([1])
    free = np.array([True, True])
    _, X = KO.attention_output(Q, K, Vr, idx, pos, True)
    np.testing.assert_allclose(X[0], [p, 1 - p], rtol=1e-14)
    jv = KO.key_jvp(Q, X, Vr, np.array([[1.0], [0.0]]), free)
    np.testing.assert_allclose(jv[0, 0], d1, rtol=1e-13)
    jv = KO.key_jvp(Q, X, Vr, np.array([[0.0], [1.0]]), free)
    np.testing.assert_allclose(jv[0, 0], -d1, rtol=1e-13)
    # with one free key and lambda_k the dual solution is a scalar ridge:
    # alpha = e / (d1^2 + lambda), dk1 = d1 alpha
    lam, Y = 0.3, np.array([[1.25]])
    e = Y[0, 0] - (p * v1 + (1 - p) * v2)
    r = KO.key_step(Q, K, K, Vr, Y, idx, pos, np.array([False, True]), lam, True)
    np.testing.assert_allclose(r["dK"][0, 0], d1 * e / (d1 * d1 + lam), rtol=1e-12)
    assert r["dK"][1, 0] == 0.0


@pytest.mark.parametrize("seed,perturb", [(4, 0.0), (5, 0.3), (6, 0.3)])
def test_dual_equals_primal_with_explicit_jacobian(seed, perturb):
    # Eq. 10 (dual) against the normal equations over the cd key entries
    Q, K0, Kc, Vr, Y, idx, pos, F, causal = _problem(seed, perturb=perturb)
    lam = 5e-2
    prim = KO.key_primal(Q, K0, Kc, Vr, Y, idx, pos, F, lam, causal)
    dual_cg = KO.key_step(Q, K0, Kc, Vr, Y, idx, pos, F, lam, causal)
    dual_dense = KO.key_step(Q, K0, Kc, Vr, Y, idx, pos, F, lam, causal, solver="dense")
    np.testing.assert_allclose(dual_cg["Kstar"], prim, atol=1e-10)
    np.testing.assert_allclose(dual_dense["Kstar"], prim, atol=1e-10)
    assert np.array_equal(dual_cg["Kstar"][F], K0[F])


def test_local_ridge_optimality_conditions():
    # gradient of ||e - J dK||^2 + lam ||dK + g||^2 vanishes at dK = K* - K_cur
    Q, K0, Kc, Vr, Y, idx, pos, F, causal = _problem(7, perturb=0.2)
    lam = 2e-2
    free = ~F
    r = KO.key_step(Q, K0, Kc, Vr, Y, idx, pos, F, lam, causal)
    X = r["X"]
    delta = np.where(free[:, None], r["Kstar"] - Kc, 0.0)
    g = np.where(free[:, None], Kc - K0, 0.0)
    res = KO.key_jvp(Q, X, Vr, delta, free) - r["E"]
    grad = KO.key_vjp(Q, X, Vr, res, free) + lam * np.where(free[:, None], delta + g, 0.0)
    assert np.abs(grad).max() < 1e-10


def test_limits_in_lambda_and_zero_residual():
    Q, K0, Kc, Vr, Y, idx, pos, F, causal = _problem(8)
    # lambda_k -> infinity keeps the keys
    r = KO.key_step(Q, K0, K0, Vr, Y, idx, pos, F, 1e12, causal)
    assert np.abs(r["Kstar"] - K0).max() < 1e-10
    # a target the retained cache already reproduces gives alpha = 0, K* = K0
    Y0 = _f(Q, K0, Vr, idx, pos, causal)
    r = KO.key_step(Q, K0, K0, Vr, Y0, idx, pos, F, 1e-2, causal)
    assert np.abs(r["Kstar"] - K0).max() < 1e-12
    # every token fixed: nothing moves
    r = KO.key_step(Q, K0, K0, Vr, Y, idx, pos, np.ones_like(F), 1e-2, causal)
    assert np.array_equal(r["Kstar"], K0)


def test_small_step_decreases_the_nonlinear_objective():
    # with a small residual the linearization is accurate, so the key step
    # lowers the true objective ||Y - f(K)||^2 + lam ||K - K0||^2
    Q, K0, Kc, Vr, Y, idx, pos, F, causal = _problem(9, scale=0.5)
    f0 = _f(Q, K0, Vr, idx, pos, causal)
    rng = np.random.default_rng(10)
    Yt = f0 + 0.05 * rng.standard_normal(f0.shape)
    lam = 1e-2
    r = KO.key_step(Q, K0, K0, Vr, Yt, idx, pos, F, lam, causal)
    before = np.sum((Yt - f0) ** 2)
    after = np.sum((Yt - _f(Q, r["Kstar"], Vr, idx, pos, causal)) ** 2) + lam * np.sum((r["Kstar"] - K0) ** 2)
    assert after < before


def test_equivariant_under_slot_permutation():
    Q, K0, Kc, Vr, Y, idx, pos, F, causal = _problem(11)
    r = KO.key_step(Q, K0, K0, Vr, Y, idx, pos, F, 1e-2, causal, solver="dense")
    perm = np.random.default_rng(12).permutation(K0.shape[0])
    rp = KO.key_step(Q, K0[perm], K0[perm], Vr[perm], Y, idx[perm], pos, F[perm], 1e-2, causal,
                     solver="dense")
    np.testing.assert_allclose(rp["Kstar"], r["Kstar"][perm], atol=1e-11)


def test_conjugate_gradient_on_a_known_system():
    rng = np.random.default_rng(13)
    A = rng.standard_normal((30, 30))
    A = A @ A.T + 0.5 * np.eye(30)
    b = rng.standard_normal(30)
    x, it, rel = KO.conjugate_gradient(lambda v: A @ v, b, tol=1e-13, max_iter=200)
    np.testing.assert_allclose(x, np.linalg.solve(A, b), atol=1e-10)
    assert rel <= 1e-13 and it <= 200


def test_workload_unit_value_step_residual_feeds_the_key_step():
    # at S = 1 the key step starts from the value step's result, where
    # Y - X V* = lambda_v Z, so E = lambda_v Z (App. D.1)
    cfg = W.config(1)
    q, K, V, _ = W.make_unit(cfg, 0, 0)
    qd, Kd, Vd = (W.decode(a, cfg.dtype) for a in (q, K, V))
    r = KO.grkv_unit(qd, Kd, Vd, cfg.window, cfg.budget, cfg.pool_kernel, cfg.lam, cfg.lam)
    np.testing.assert_allclose(r["key"]["E"], cfg.lam * r["Z"], atol=1e-13)
    assert r["key"]["rel_residual"] <= 1e-12
    assert np.array_equal(r["Kstar"][r["fixed"]], r["K0"][r["fixed"]])
    assert np.abs(r["Kstar"] - r["K0"]).max() > 0


# ------------------------------------------------------ alternating steps ----

def _unit(cfg_id=1, **over):
    cfg = W.config(cfg_id, **over)
    q, K, V, _ = W.make_unit(cfg, 0, 1)
    return cfg, tuple(W.decode(a, cfg.dtype) for a in (q, K, V))


def test_one_alternating_step_is_the_value_and_key_step():
    cfg, (qd, Kd, Vd) = _unit()
    a = KO.grkv_alternating(qd, Kd, Vd, cfg.window, cfg.budget, cfg.pool_kernel, cfg.lam,
                            cfg.lam, steps=1)
    b = KO.grkv_unit(qd, Kd, Vd, cfg.window, cfg.budget, cfg.pool_kernel, cfg.lam, cfg.lam)
    assert a["steps_run"] == 1
    np.testing.assert_allclose(a["Kstar"], b["Kstar"], atol=1e-12)
    np.testing.assert_allclose(a["Vstar"], b["Vstar"], atol=1e-12)


def test_second_step_linearizes_at_the_moved_keys():
    # step 2 must use G = K^(1) - K0: its right-hand side is E + J_G G, and its
    # key update solves the local ridge problem around K^(1) (KKT of Eq. 9-10
    # with the g term), checked against the explicit-Jacobian primal
    cfg, (qd, Kd, Vd) = _unit(n=256, budget=48)
    lam = 5e-2
    a = KO.grkv_alternating(qd, Kd, Vd, cfg.window, cfg.budget, cfg.pool_kernel, lam, lam,
                            steps=2, stop=0.0)
    assert a["steps_run"] == 2
    h1, h2 = a["history"]
    K1, V2 = h1["Kstar"], h2["Vstar"]
    prim = KO.key_primal(a["Q"], a["K0"], K1, V2, a["Y"], a["idx"], a["pos"], a["fixed"], lam)
    np.testing.assert_allclose(h2["Kstar"], prim, atol=1e-9)
    # the second value step is the ridge solution for X at K^(1), anchored at V0
    X1 = KO.attention_output(a["Q"], K1, V2, a["idx"], a["pos"], True)[1]
    G = np.flatnonzero(~a["fixed"])
    A = np.vstack([X1[:, G], np.sqrt(lam) * np.eye(G.size)])
    b = np.vstack([a["Y"] - X1 @ a["V0"], np.zeros((G.size, a["Y"].shape[1]))])
    dVG = np.linalg.lstsq(A, b, rcond=None)[0]
    np.testing.assert_allclose(V2[G] - a["V0"][G], dVG, atol=1e-9)
    assert np.array_equal(V2[a["fixed"]], a["V0"][a["fixed"]])


def test_stop_rule_when_keys_cannot_move():
    # lambda_k -> infinity keeps K = K0, so the second value step repeats the
    # first and the iterates stop changing: the loop ends after step 2
    cfg, (qd, Kd, Vd) = _unit()
    a = KO.grkv_alternating(qd, Kd, Vd, cfg.window, cfg.budget, cfg.pool_kernel, cfg.lam,
                            1e14, steps=5)
    assert a["steps_run"] == 2
    assert a["history"][1]["delta_v"] <= 1e-9 and a["history"][1]["delta_k"] <= 1e-9
    assert np.abs(a["Kstar"] - a["K0"]).max() < 1e-10
