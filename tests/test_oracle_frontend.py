"""Pins for the budget front-end oracle: the pyramid schedule by its closed
form and invariants, the adaptive allocation by brute force and by the tie
rule, and the ragged compression against the per-unit oracle."""
import itertools

import numpy as np
import pytest

import workloads as W
from oracle import grkv_frontend_oracle as FO
from oracle import grkv_oracle as O


def test_pyramid_schedule():
    b = FO.pyramid_budgets(32, 8, 2048, 32, 32768)
    per = b.reshape(32, 8)
    assert np.all(per == per[:, :1])                    # heads of a layer share it
    assert per[:, 0].sum() == 32 * 2048                 # the mean is kept
    assert np.all(np.diff(per[:, 0]) <= 0)              # falls with depth
    assert abs(per[-1, 0] - 1024) <= 1 and abs(per[0, 0] - 3072) <= 1
    # linear: constant step up to rounding
    steps = -np.diff(per[:, 0])
    assert steps.max() - steps.min() <= 2
    assert np.array_equal(FO.pyramid_budgets(1, 4, 500, 16, 1000), np.full(4, 500))
    # clipping at the window keeps every budget in [w, n]
    b = FO.pyramid_budgets(4, 1, 40, 32, 100, ratio=0.1)
    assert np.all(b >= 32) and np.all(b <= 100)


def _brute_adaptive(pooled, H, c, w):
    U, P = pooled.shape
    out = []
    for l in range(U // H):
        items = [(-float(pooled[l * H + h, j]), h, j) for h in range(H) for j in range(P)]
        items.sort()
        taken = [0] * H
        for _, h, _ in items[:H * (c - w)]:
            taken[h] += 1
        out += [w + t for t in taken]
    return np.array(out)


@pytest.mark.parametrize("seed", range(3))
def test_adaptive_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    H, P, c, w = 3, 7, 5, 2
    pooled = rng.integers(0, 4, size=(2 * H, P)).astype(np.float64)   # many ties
    got = FO.adaptive_budgets(pooled, 2, H, c, w)
    np.testing.assert_array_equal(got, _brute_adaptive(pooled, H, c, w))
    assert np.all(got.reshape(2, H).sum(axis=1) == H * c)


def test_adaptive_tie_rule_and_extremes():
    H, P, c, w = 4, 6, 5, 1
    # all scores equal: the lower heads fill first, P tokens each
    got = FO.adaptive_budgets(np.ones((H, P)), 1, H, c, w)
    k = H * (c - w)
    want = [w + min(P, max(0, k - h * P)) for h in range(H)]
    np.testing.assert_array_equal(got, want)
    # one head holds every large score: it takes up to its P tokens
    pooled = np.zeros((H, P))
    pooled[2] = 10.0
    got = FO.adaptive_budgets(pooled, 1, H, c, w)
    assert got[2] == w + min(P, k) and got.sum() == H * c


def test_ragged_units_match_the_uniform_oracle():
    cfg = W.config(1)
    q, K, V = W.make_batch(cfg)
    dec = [W.decode(a, cfg.dtype) for a in (q, K, V)]
    res = FO.compress_ragged(*dec, [96, 128], cfg.window, cfg.pool_kernel, cfg.lam)
    for u, b in enumerate([96, 128]):
        r = O.compress_unit(dec[0][u], dec[1][u], dec[2][u], cfg.window, b, cfg.pool_kernel, cfg.lam)
        assert np.array_equal(res[u]["idx"], r["idx"]) and res[u]["idx"].size == b
        np.testing.assert_array_equal(res[u]["Vstar"], r["Vstar"])
    np.testing.assert_array_equal(FO.packed_offsets([96, 128, 5]), [0, 96, 224])


def _h2o_brute(q_all, K):
    # plain loops over rows and keys: each row's causal softmax, then column sums
    G, n, d = q_all.shape
    s = [0.0] * n
    for g in range(G):
        for i in range(n):
            logits = [sum(q_all[g, i, e] * K[j, e] for e in range(d)) / d ** 0.5 for j in range(i + 1)]
            mx = max(logits)
            ex = [np.exp(x - mx) for x in logits]
            z = sum(ex)
            for j in range(i + 1):
                s[j] += ex[j] / z
    return np.array(s)


def test_h2o_scores_brute_force():
    rng = np.random.default_rng(3)
    G, n, d, w = 2, 11, 4, 3
    q = rng.standard_normal((G, n, d))
    K = rng.standard_normal((n, d))
    want = _h2o_brute(q, K)
    np.testing.assert_allclose(FO.h2o_scores(q, K, w, all_columns=True), want, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(FO.h2o_scores(q, K, w), want[: n - w], rtol=1e-12, atol=1e-14)


def test_h2o_scores_closed_forms():
    G, n, d, w = 3, 50, 8, 4
    K = np.random.default_rng(4).standard_normal((n, d))
    # zero queries: row i spreads 1/(i+1) over keys 0..i, so
    # s_j = G * (H_n - H_j) with H_k the k-th harmonic number
    s = FO.h2o_scores(np.zeros((G, n, d)), K, w, all_columns=True)
    H = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, n + 1))])
    np.testing.assert_allclose(s, G * (H[n] - H[:n]), rtol=1e-13)
    # every row is a distribution: the column sums over all keys total G * n
    q = np.random.default_rng(5).standard_normal((G, n, d))
    assert abs(FO.h2o_scores(q, K, w, all_columns=True).sum() - G * n) < 1e-9
    # a key every query points at takes nearly all the mass of the rows that see it
    q = np.tile(40.0 * K[7] / np.linalg.norm(K[7]), (G, n, 1))
    s = FO.h2o_scores(q, K, w, all_columns=True)
    assert s[7] > 0.99 * G * (n - 7)


def test_h2o_compress_uses_the_scores():
    # the retained prefix tokens are the top c - w by accumulated attention
    # (no pooling), and the merge is the value step on the window queries
    rng = np.random.default_rng(6)
    G, n, d, w, c = 2, 80, 8, 4, 20
    q_all = rng.standard_normal((G, n, d))
    K, Vv = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    q_obs = q_all[:, n - w:, :]
    r = FO.compress_h2o(q_all, q_obs, K, Vv, w, c, 1e-2)
    s = FO.h2o_scores(q_all, K, w)
    top = np.sort(np.lexsort((np.arange(n - w), -s))[: c - w])
    np.testing.assert_array_equal(r["idx"], np.concatenate([top, np.arange(n - w, n)]))
    np.testing.assert_array_equal(r["s"], s)
    # the fixed top-beta subset follows the same (accumulated-attention) order
    base = O.compress_unit(q_obs, K, Vv, w, c, 1, 1e-2, idx=r["idx"], scores=s)
    np.testing.assert_allclose(r["Vstar"], base["Vstar"], atol=1e-12)
