"""Pins for the oracle's SnapKV-style span retention and fixed-token set.

SnapKV scores prefix tokens by the window's attention, pools the scores over
segments and keeps the top-k (Sec. 1, Sec. 2); the fixed set is the sinks, the
window and the top beta of the retained tokens (Sec. 3.4; App. D.3).
"""
import math

import numpy as np
import pytest

from oracle import grkv_oracle as O


def test_pool_box_matches_convolution_and_delta():
    rng = np.random.default_rng(0)
    s = rng.random(57)
    for k in (1, 3, 7, 9):
        want = np.convolve(s, np.ones(k), mode="same")   # library reference
        np.testing.assert_allclose(O.pool_box(s, k), want, rtol=0, atol=1e-14)
    # a single spike spreads into a box of width k, clipped at the ends
    for t in (0, 2, 30, 56):
        e = np.zeros(57)
        e[t] = 1.0
        p = O.pool_box(e, 7)
        want = np.zeros(57)
        want[max(0, t - 3): t + 4] = 1.0
        np.testing.assert_array_equal(p, want)
    with pytest.raises(AssertionError):
        O.pool_box(s, 4)


def test_selection_order_brute_force_with_ties():
    rng = np.random.default_rng(1)
    p = rng.integers(0, 6, size=200).astype(float)   # many exact ties
    want = sorted(range(200), key=lambda j: (-p[j], j))
    np.testing.assert_array_equal(O.selection_order(p), want)


def test_zero_query_closed_form_selection():
    # Q = 0: every prefix score is sum_r 1/(pos_r + 1), constant in j, so the
    # pooled score is maximal and tied on the interior [h, P - h); the tie rule
    # keeps the lowest interior positions.
    G, w, d, n, k = 2, 4, 8, 64, 7
    h = (k - 1) // 2
    rng = np.random.default_rng(2)
    q = np.zeros((G, w, d))
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    for budget in (w, w + 1, w + 13, w + (n - w) - 2 * h):
        r = O.compress_unit(q, K, V, w, budget, k, 1e-2)
        sel = budget - w
        want = np.concatenate([np.arange(h, h + sel), np.arange(n - w, n)])
        np.testing.assert_array_equal(r["idx"], want)
        const = sum(1.0 / (p + 1) for p in O.query_positions(G, w, n))
        np.testing.assert_allclose(r["s"], const, rtol=1e-13)


def test_planted_span_is_retained():
    # Keys of one span share the query direction; the span and its pooled
    # neighbourhood must be the first picks.
    G, w, d, n, k = 1, 4, 16, 200, 5
    rng = np.random.default_rng(3)
    K = rng.standard_normal((n, d))
    V = rng.standard_normal((n, d))
    u = rng.standard_normal(d)
    u /= np.linalg.norm(u)
    K[100:110] += 4.0 * u
    q = np.broadcast_to(3.0 * u, (G, w, d)).copy()
    r = O.compress_unit(q, K, V, w, w + 10, k, 1e-2)
    assert set(range(100, 110)) <= set(r["order"][:14].tolist())
    assert set(r["idx"][:-w].tolist()) <= set(range(98, 112))


def test_duplicated_query_head_changes_nothing():
    # Two identical query heads double every score: same selection as one head.
    w, d, n, k = 4, 8, 80, 7
    rng = np.random.default_rng(4)
    q1 = rng.standard_normal((1, w, d))
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    r1 = O.compress_unit(q1, K, V, w, 24, k, 1e-2)
    r2 = O.compress_unit(np.concatenate([q1, q1]), K, V, w, 24, k, 1e-2)
    np.testing.assert_allclose(r2["s"], 2 * r1["s"], rtol=1e-13)
    np.testing.assert_array_equal(r1["idx"], r2["idx"])


def test_retained_index_shape_and_window():
    rng = np.random.default_rng(5)
    G, w, d, n = 2, 6, 8, 100
    q = rng.standard_normal((G, w, d))
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    for budget in (w, 7, 30, n):
        r = O.compress_unit(q, K, V, w, budget, 7, 1e-2)
        idx = r["idx"]
        assert idx.shape == (budget,)
        assert np.all(np.diff(idx) > 0)
        np.testing.assert_array_equal(idx[-w:], np.arange(n - w, n))
        np.testing.assert_array_equal(r["K0"], K[idx])


def test_fixed_mask_hand_case():
    # n = 20, w = 3, c = 10: prefix order given; beta = 0.25 -> floor(2.5) = 2
    # top picks fixed; sinks below 4 fixed when retained; window fixed.
    n, w, c = 20, 3, 10
    order = np.array([9, 2, 15, 5, 11, 0, 7, 13, 1, 3, 4, 6, 8, 10, 12, 14, 16])
    idx = O.retained_index(order, n, w, c)
    np.testing.assert_array_equal(idx, [0, 2, 5, 7, 9, 11, 15, 17, 18, 19])
    F = O.fixed_mask(idx, order, n, w, c, O.Options(n_sink=4, beta=0.25))
    want = {0: True, 2: True, 5: False, 7: False, 9: True, 11: False, 15: False,
            17: True, 18: True, 19: True}
    assert dict(zip(idx.tolist(), F.tolist())) == want
    F2 = O.fixed_mask(idx, order, n, w, c, O.Options(n_sink=0, beta=0.0, fix_window=False))
    assert not F2.any()
    F3 = O.fixed_mask(idx, order, n, w, c, O.Options(beta=1.0))
    assert F3.all()


def test_beta_count_uses_float32_beta():
    # the ABI carries beta as float32; 0.1f * 2048 = 204.8000031 -> 204
    opt = O.Options(beta=0.1)
    assert math.floor(opt.beta * 2048) == 204
    assert math.floor(opt.beta * 512) == 51
    assert math.floor(opt.beta * 128) == 12
