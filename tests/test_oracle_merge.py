"""Pins for the oracle's value step (Eq. 6-8; Algorithm 1 value step; App. D.1
primal and dual; App. D.3 fixed tokens).

The value step minimises ||Y - X V||_F^2 + lambda ||V - V0||_F^2 over the free
rows V_G with V_F = V0_F.  Each test checks the oracle against the mathematics
of that problem: an independent least-squares solve, the optimality
conditions, and limits the paper states or implies.
"""
import math

import numpy as np
import pytest

from oracle import grkv_oracle as O


def _problem(seed, m=6, c=15, d=4, n_fixed=3):
    rng = np.random.default_rng(seed)
    X = rng.random((m, c))
    X /= X.sum(axis=1, keepdims=True)          # rows of a softmax
    Y = rng.standard_normal((m, d))
    V0 = rng.standard_normal((c, d))
    F = np.zeros(c, dtype=bool)
    F[rng.choice(c, n_fixed, replace=False)] = True
    return X, Y, V0, F


@pytest.mark.parametrize("lam", [1e-2, 1e-1, 1.0])
def test_dual_matches_augmented_least_squares(lam):
    # min ||R - X_G dV_G||^2 + lam ||dV_G||^2  ==  lstsq([X_G; sqrt(lam) I], [R; 0])
    X, Y, V0, F = _problem(0)
    dV, Z, R, st = O.merge_dual(X, Y, V0, F, lam)
    assert st == O.STATUS_OK
    G = np.flatnonzero(~F)
    A = np.vstack([X[:, G], math.sqrt(lam) * np.eye(G.size)])
    b = np.vstack([Y - X @ V0, np.zeros((G.size, Y.shape[1]))])
    want = np.linalg.lstsq(A, b, rcond=None)[0]
    np.testing.assert_allclose(dV[G], want, atol=1e-10)
    assert np.all(dV[F] == 0.0)


@pytest.mark.parametrize("seed", range(4))
def test_primal_equals_dual(seed):
    X, Y, V0, F = _problem(seed, m=5, c=12)
    d1, *_ = O.merge_dual(X, Y, V0, F, 1e-2)
    d2 = O.merge_primal(X, Y, V0, F, 1e-2)
    np.testing.assert_allclose(d1, d2, atol=1e-10)


def test_optimality_conditions_and_residual_identity():
    lam = 3e-2
    X, Y, V0, F = _problem(1)
    dV, Z, R, _ = O.merge_dual(X, Y, V0, F, lam)
    G = np.flatnonzero(~F)
    XG = X[:, G]
    # KKT on the free rows: X_G^T (X_G dV_G - R) + lam dV_G = 0
    kkt = XG.T @ (XG @ dV[G] - R) + lam * dV[G]
    assert np.abs(kkt).max() < 1e-12
    # Y - X V* = lam Z  (from X_G X_G^T Z = R - lam Z)
    np.testing.assert_allclose(Y - X @ (V0 + dV), lam * Z, atol=1e-12)


def test_objective_is_minimised_finite_difference():
    lam = 5e-2
    X, Y, V0, F = _problem(2)
    dV, *_ = O.merge_dual(X, Y, V0, F, lam)
    Vs = V0 + dV

    def obj(V):
        return np.sum((Y - X @ V) ** 2) + lam * np.sum((V - V0) ** 2)

    f0 = obj(Vs)
    rng = np.random.default_rng(9)
    G = np.flatnonzero(~F)
    for _ in range(20):
        D = np.zeros_like(Vs)
        D[G] = rng.standard_normal((G.size, Vs.shape[1]))
        for eps in (1e-3, 1e-5):
            assert obj(Vs + eps * D) >= f0 - 1e-14
            # symmetric difference of a quadratic: gradient along D is zero
            g = (obj(Vs + eps * D) - obj(Vs - eps * D)) / (2 * eps)
            assert abs(g) < 1e-8


def test_zero_lambda_reproduces_target_exactly():
    # lambda = 0 with >= m free tokens and X_G of full row rank: the merged
    # cache reproduces the window's full-cache attention output exactly.
    X, Y, V0, F = _problem(3, m=5, c=20, n_fixed=4)
    dV, Z, R, st = O.merge_dual(X, Y, V0, F, 0.0)
    assert st == O.STATUS_OK
    np.testing.assert_allclose(X @ (V0 + dV), Y, atol=1e-10)
    assert O.discrepancy(Y, X, V0 + dV) < 1e-20


def test_zero_lambda_rank_deficient_is_flagged():
    X, Y, V0, F = _problem(4, m=6, c=8, n_fixed=4)   # only 4 free < m = 6
    _, _, _, st = O.merge_dual(X, Y, V0, F, 0.0)
    assert st == O.STATUS_SINGULAR


def test_large_lambda_keeps_values():
    X, Y, V0, F = _problem(5)
    R = Y - X @ V0
    for lam in (1e6, 1e12):
        dV, *_ = O.merge_dual(X, Y, V0, F, lam)
        # ||dV|| <= ||X_G|| ||R|| / lam
        bound = np.linalg.norm(np.where(F[None, :], 0, X), 2) * np.linalg.norm(R) / lam
        assert np.linalg.norm(dV) <= bound * (1 + 1e-9)


def test_all_fixed_keeps_values():
    X, Y, V0, _ = _problem(6)
    F = np.ones(X.shape[1], dtype=bool)
    dV, *_ = O.merge_dual(X, Y, V0, F, 1e-2)
    assert np.all(dV == 0.0)


def test_linear_in_values_and_equivariant_in_slots():
    lam = 1e-2
    X, Y, V0, F = _problem(7)
    dV, *_ = O.merge_dual(X, Y, V0, F, lam)
    dV2, *_ = O.merge_dual(X, 2.5 * Y, 2.5 * V0, F, lam)
    np.testing.assert_allclose(dV2, 2.5 * dV, atol=1e-12)
    perm = np.random.default_rng(1).permutation(X.shape[1])
    dVp, *_ = O.merge_dual(X[:, perm], Y, V0[perm], F[perm], lam)
    np.testing.assert_allclose(dVp, dV[perm], atol=1e-12)


def test_single_row_closed_form():
    # m = 1: Z = R / (sum_{j in G} x_j^2 + lam), dV_j = x_j Z for free j.
    x = np.array([[0.5, 0.2, 0.3]])
    V0 = np.array([[1.0], [2.0], [-1.0]])
    Y = np.array([[0.7]])
    F = np.array([False, True, False])
    lam = 0.1
    dV, Z, R, _ = O.merge_dual(x, Y, V0, F, lam)
    r = 0.7 - (0.5 * 1.0 + 0.2 * 2.0 + 0.3 * -1.0)
    z = r / (0.25 + 0.09 + lam)
    np.testing.assert_allclose(R, [[r]], atol=1e-15)
    np.testing.assert_allclose(dV[:, 0], [0.5 * z, 0.0, 0.3 * z], atol=1e-15)


def test_full_budget_has_nothing_to_merge():
    # c = n keeps every token: X equals the full attention, so R = 0 and V* = V0.
    rng = np.random.default_rng(8)
    G, w, d, n = 2, 4, 8, 50
    q = rng.standard_normal((G, w, d))
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    r = O.compress_unit(q, K, V, w, n, 7, 1e-2)
    np.testing.assert_array_equal(r["idx"], np.arange(n))
    assert np.abs(r["R"]).max() < 1e-14
    np.testing.assert_allclose(r["Vstar"], V, atol=1e-14)
    assert r["D_before"] < 1e-28 and r["D_after"] < 1e-28


def test_zero_lambda_full_budget_reproduces_attention():
    # zero regularisation with every token free reproduces full-cache attention
    rng = np.random.default_rng(10)
    G, w, d, n = 1, 3, 6, 30
    q = rng.standard_normal((G, w, d))
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    opt = O.Options(n_sink=0, beta=0.0, fix_window=False)
    r = O.compress_unit(q, K, V, w, 12, 7, 0.0, opt)
    assert r["status"] == O.STATUS_OK
    np.testing.assert_allclose(r["X"] @ r["Vstar"], r["Y"], atol=1e-10)
    assert r["D_after"] < 1e-18 < r["D_before"]


def test_end_to_end_tiny_config_properties():
    import workloads as W
    cfg = W.config(1)
    q, K, V = W.make_batch(cfg)
    qd, Kd, Vd = (W.decode(a, cfg.dtype) for a in (q, K, V))
    idx, k_out, v_out, st = O.compress(qd, Kd, Vd, cfg.window, cfg.budget,
                                       cfg.pool_kernel, cfg.lam)
    assert idx.shape == (2, 128) and v_out.shape == (2, 128, 64)
    for u in range(2):
        np.testing.assert_array_equal(k_out[u], Kd[u][idx[u]])
        assert st[u, 3] == 0
        assert 0 <= st[u, 2] < st[u, 1]      # the merge lowers the discrepancy
    r = O.compress_unit(qd[0], Kd[0], Vd[0], cfg.window, cfg.budget, cfg.pool_kernel,
                        cfg.lam, with_primal=True)
    np.testing.assert_allclose(r["dV"], r["dV_primal"], atol=1e-10)
    # salient spans drive the selection: span tokens are retained at several
    # times the rate of prefix tokens overall
    _, _, _, spans = W.make_unit(cfg, 0, 0)
    span_tok = set(np.concatenate([np.arange(s, s + l) for s, l in spans]).tolist())
    span_rate = len(span_tok & set(idx[0].tolist())) / len(span_tok)
    base_rate = (cfg.budget - cfg.window) / (cfg.n - cfg.window)
    assert span_rate > 3 * base_rate


@pytest.mark.parametrize("seed,lam", [(0, 1e-2), (1, 0.3), (11, 2.0)])
def test_discrepancy_closed_forms(seed, lam):
    # Eq. 4 normalised by the target energy.  Before the merge the residual is
    # R = Y - X V0, so D_before = ||R||^2 / ||Y||^2.  After it, Y - X V* = lam Z
    # (App. D.1: X_G X_G^T Z = R - lam Z), so D_after = lam^2 ||Z||^2 / ||Y||^2.
    X, Y, V0, F = _problem(seed)
    dV, Z, R, _ = O.merge_dual(X, Y, V0, F, lam)
    y2 = float(np.sum(Y ** 2))
    np.testing.assert_allclose(O.discrepancy(Y, X, V0), np.sum(R ** 2) / y2, rtol=1e-12)
    np.testing.assert_allclose(O.discrepancy(Y, X, V0 + dV), lam ** 2 * np.sum(Z ** 2) / y2,
                               rtol=1e-9)


def test_discrepancy_hand_values():
    # worked by hand: Y = [3, 4] has ||Y||^2 = 25
    Y = np.array([[3.0, 4.0]])
    X = np.array([[1.0]])
    assert O.discrepancy(Y, X, np.array([[0.0, 0.0]])) == 1.0          # 25 / 25
    assert O.discrepancy(Y, X, np.array([[3.0, 0.0]])) == 16.0 / 25.0  # (0^2 + 4^2) / 25
    assert O.discrepancy(Y, X, Y) == 0.0
    # two rows, two retained slots: X V = [[1.5, 0], [0, 2]] against Y = [[1, 0], [0, 1]]
    Y2 = np.eye(2)
    X2 = np.array([[0.5, 0.5], [0.0, 1.0]])
    V2 = np.array([[1.0, -2.0], [2.0, 2.0]])
    # X2 V2 = [[1.5, 0.0], [2.0, 2.0]]; residual [[-0.5, 0], [-2, -1]] -> 0.25 + 4 + 1 = 5.25
    assert O.discrepancy(Y2, X2, V2) == 5.25 / 2.0


def test_discrepancy_single_row_merge_by_hand():
    # the m = 1 case of test_single_row_closed_form, carried through to D:
    # D_before = r^2 / y^2 and D_after = (lam z)^2 / y^2 with z = r / (sum_G x^2 + lam)
    x = np.array([[0.5, 0.2, 0.3]])
    V0 = np.array([[1.0], [2.0], [-1.0]])
    Y = np.array([[0.7]])
    F = np.array([False, True, False])
    lam = 0.1
    dV, Z, R, _ = O.merge_dual(x, Y, V0, F, lam)
    r = 0.7 - 0.6
    z = r / (0.25 + 0.09 + lam)
    np.testing.assert_allclose(O.discrepancy(Y, x, V0), r * r / 0.49, rtol=1e-12)
    np.testing.assert_allclose(O.discrepancy(Y, x, V0 + dV), (lam * z) ** 2 / 0.49, rtol=1e-12)
