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
