"""Pins for the oracle's window attention (Sec. 3.1 standard attention; Eq. 4
window target Y = softmax(Q K^T / sqrt(d)) V).

Each check is fixed by something other than the oracle's own formula: a closed
form, brute force in plain Python, or an invariant of softmax attention.
"""
import math

import numpy as np
import pytest

from oracle import grkv_oracle as O


def _rand(seed, *shape):
    return np.random.default_rng(seed).standard_normal(shape)


def test_zero_query_is_uniform_over_visible_keys():
    # Q = 0 => every visible logit is 0 => row at position p averages V[0..p]
    # and its log-sum-exp is log(p + 1).
    G, w, d, n = 2, 5, 8, 40
    K, V = _rand(1, n, d), _rand(2, n, d)
    Q = np.zeros((G * w, d))
    pos = O.query_positions(G, w, n)
    A, lse = O.softmax_rows(O.window_logits(Q, K, pos, causal=True))
    Y = A @ V
    for r in range(G * w):
        p = pos[r]
        np.testing.assert_allclose(Y[r], V[: p + 1].mean(axis=0), rtol=0, atol=1e-13)
        assert abs(lse[r] - math.log(p + 1)) < 1e-13
    # without the causal rule every row averages all n keys
    A2, lse2 = O.softmax_rows(O.window_logits(Q, K, pos, causal=False))
    np.testing.assert_allclose(A2 @ V, np.broadcast_to(V.mean(axis=0), (G * w, d)), atol=1e-13)
    np.testing.assert_allclose(lse2, math.log(n), atol=1e-13)


def test_brute_force_python_loops():
    # Plain-Python attention on a tiny case, different evaluation order
    # (no max shift, explicit double loops).
    G, w, d, n = 2, 3, 4, 9
    rng = np.random.default_rng(3)
    q = rng.standard_normal((G, w, d))
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    Q = O.stack_queries(q)
    pos = O.query_positions(G, w, n)
    A, lse = O.softmax_rows(O.window_logits(Q, K, pos, causal=True))
    for g in range(G):
        for i in range(w):
            r = g * w + i
            p = n - w + i
            e = [math.exp(sum(q[g, i, t] * K[j, t] for t in range(d)) / math.sqrt(d))
                 for j in range(p + 1)]
            z = sum(e)
            assert abs(lse[r] - math.log(z)) < 1e-12
            for j in range(n):
                want = e[j] / z if j <= p else 0.0
                assert abs(A[r, j] - want) < 1e-14
            y = [sum(e[j] * V[j, t] for j in range(p + 1)) / z for t in range(d)]
            np.testing.assert_allclose((A @ V)[r], y, atol=1e-13)


def test_dominant_key_picks_its_value():
    # A query aligned 60x with one key's direction puts ~all mass on that key.
    d, n = 16, 30
    rng = np.random.default_rng(4)
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    K /= np.linalg.norm(K, axis=1, keepdims=True)
    j = 11
    Q = (60.0 * math.sqrt(d)) * K[j][None, :]
    A, _ = O.softmax_rows(O.window_logits(Q, K, np.array([n - 1]), causal=True))
    assert A[0, j] > 1 - 1e-9
    np.testing.assert_allclose((A @ V)[0], V[j], atol=1e-8)


def test_common_key_offset_does_not_change_attention():
    # Adding the same vector to every key shifts each row's logits by a
    # constant, which softmax ignores.
    G, w, d, n = 1, 4, 8, 25
    Q, K = _rand(5, G * w, d), _rand(6, n, d)
    a = _rand(7, d)
    pos = O.query_positions(G, w, n)
    A1, lse1 = O.softmax_rows(O.window_logits(Q, K, pos, True))
    A2, lse2 = O.softmax_rows(O.window_logits(Q, K + a, pos, True))
    np.testing.assert_allclose(A1, A2, atol=1e-14)
    # LSE shifts only where every visible key moved, i.e. by q.a/sqrt(d)
    np.testing.assert_allclose(lse2 - lse1, Q @ a / math.sqrt(d), atol=1e-12)


def test_causal_rule_hides_later_keys():
    G, w, d, n = 2, 4, 8, 20
    Q, K, V = _rand(8, G * w, d), _rand(9, n, d), _rand(10, n, d)
    pos = O.query_positions(G, w, n)
    A, _ = O.softmax_rows(O.window_logits(Q, K, pos, True))
    Y = A @ V
    K2, V2 = K.copy(), V.copy()
    K2[n - 2:] += 5.0
    V2[n - 2:] -= 3.0
    A2, _ = O.softmax_rows(O.window_logits(Q, K2, pos, True))
    Y2 = A2 @ V2
    for r in range(G * w):
        if pos[r] < n - 2:
            np.testing.assert_allclose(Y[r], Y2[r], atol=1e-14)
        else:
            assert np.abs(Y[r] - Y2[r]).max() > 1e-3
    assert np.all(A[pos == n - w][:, n - w + 1:] == 0.0)


def test_query_stacking_matches_single_head():
    # Stacked row g*w + i must equal head g computed on its own.
    G, w, d, n = 3, 4, 8, 30
    rng = np.random.default_rng(11)
    q = rng.standard_normal((G, w, d))
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    Q = O.stack_queries(q)
    pos = O.query_positions(G, w, n)
    A, _ = O.softmax_rows(O.window_logits(Q, K, pos, True))
    for g in range(G):
        Qg = q[g]
        pg = np.arange(n - w, n)
        Ag, _ = O.softmax_rows(O.window_logits(Qg, K, pg, True))
        np.testing.assert_array_equal(A[g * w:(g + 1) * w], Ag)
