"""Pins for the carrier-concentration oracle (App. B, "Quantitative Carrier
Concentration"; Sec. 1 on span boundaries as carriers).

The assignment is checked by brute force and by invariances of the cosine
similarity; the metrics by closed forms on constructed loads."""
import math

import numpy as np
import pytest

from oracle import grkv_carrier_oracle as C


def _brute_assign(K, idx):
    n = K.shape[0]
    out = np.full(n, -1)
    for j in range(n):
        if j in set(idx.tolist()):
            continue
        best, bs = -np.inf, -1
        for s, i in enumerate(idx):
            nj, ni = np.linalg.norm(K[j]), np.linalg.norm(K[i])
            cs = float(K[j] @ K[i]) / (nj * ni) if nj > 0 and ni > 0 else 0.0
            if cs > best:          # strict: the first (lowest) slot keeps a tie
                best, bs = cs, s
        out[j] = bs
    return out


@pytest.mark.parametrize("seed", range(3))
def test_assignment_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    n, d = 60, 5
    K = rng.standard_normal((n, d))
    idx = np.sort(rng.choice(n, 17, replace=False))
    np.testing.assert_array_equal(C.carrier_assignment(K, idx), _brute_assign(K, idx))


def test_assignment_is_scale_invariant_and_ties_go_low():
    rng = np.random.default_rng(4)
    K = rng.standard_normal((40, 6))
    idx = np.array([3, 9, 10, 11, 30])
    a = C.carrier_assignment(K, idx)
    scale = rng.uniform(0.1, 10.0, size=(40, 1))
    np.testing.assert_array_equal(C.carrier_assignment(K * scale, idx), a)
    # two retained keys along the same direction tie for every evicted token:
    # the lower slot wins
    K2 = K.copy()
    K2[11] = 3.0 * K2[9]
    a2 = C.carrier_assignment(K2, idx)
    assert not np.any(a2 == 3)   # slot 3 (position 11) never beats slot 1 (position 9)
    # a zero evicted key has cosine 0 with all: slot 0 unless some cosine is positive
    K3 = -np.abs(K)
    K3[0] = 0.0
    assert C.carrier_assignment(K3, idx)[0] == 0


def test_metrics_closed_forms():
    idx = np.array([0, 1, 2, 3, 10, 11, 20, 30])   # runs: [0..3], [10, 11], [20], [30]
    c = idx.size
    bnd = np.array([1, 0, 0, 1, 1, 1, 1, 1], dtype=bool)
    # uniform load: b = b_eff = c, A_max = 1, Gini = 0
    assign = np.repeat(np.arange(c), 3)
    m = C.carrier_metrics(assign, idx)
    assert m["b"] == c and math.isclose(m["b_eff"], c) and math.isclose(m["a_max"], 1.0)
    assert m["gini"] == 0.0
    assert math.isclose(m["boundary_fraction"], bnd.sum() / c)
    assert math.isclose(m["enrichment"], 1.0) and math.isclose(m["boundary_interior_load"], 1.0)
    # everything on one carrier: b = b_eff = 1, A_max = c, Gini = 1 - 1/c
    m = C.carrier_metrics(np.full(50, 5), idx)
    assert m["b"] == 1 and math.isclose(m["b_eff"], 1.0) and math.isclose(m["a_max"], c)
    assert math.isclose(m["gini"], 1.0 - 1.0 / c)
    assert math.isclose(m["boundary_share"], 1.0)   # slot 5 (position 11) ends a run
    assert math.isinf(m["boundary_interior_load"])
    # loads (1, 3) on two slots of a two-slot run: Gini = |1-3| * 2 / (2 * 2 * 4) = 1/4
    m = C.carrier_metrics(np.array([0, 1, 1, 1]), np.array([7, 8]))
    assert math.isclose(m["gini"], 0.25) and math.isclose(m["b_eff"], 16 / 10)
    assert math.isnan(m["boundary_interior_load"])   # no interior slot


def test_l_common_against_the_value_step_closed_form():
    # for merged values Y - X V* = lambda Z (App. D.1), so the compressed-cache
    # discrepancy of each unit is lambda^2 ||Z||^2, independently of X V*
    import workloads as W
    from oracle import grkv_oracle as O
    cfg = W.config(1)
    yf, yc, num, den = [], [], 0.0, 0.0
    for head in range(2):
        q, K, V, _ = W.make_unit(cfg, 0, head)
        r = O.compress_unit(*(W.decode(a, cfg.dtype) for a in (q, K, V)), cfg.window, cfg.budget,
                            cfg.pool_kernel, cfg.lam)
        yf.append(r["Y"])
        yc.append(r["X"] @ r["Vstar"])
        num += cfg.lam ** 2 * float(np.sum(r["Z"] ** 2))
        den += float(np.sum(r["Y"] ** 2))
    assert math.isclose(C.l_common(yf, yc), num / den, rel_tol=1e-9)
    assert C.l_common(yf, yf) == 0.0
