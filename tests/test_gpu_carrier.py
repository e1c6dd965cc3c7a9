"""GPU parity of the carrier-concentration diagnostics (grkv_carrier_stats)
against the float64 oracle.

The assignment is an argmax of fp32 cosine similarities on the GPU and of
fp64 ones in the oracle, so where the two differ the GPU's choice must be a
near-tie: its fp64 cosine within 1e-5 of the best.  The metrics are compared
with the oracle's metrics of the GPU's own assignment (exact integer loads),
and L_common with the same sum taken from the stats in float64.
"""
import numpy as np
import pytest

import workloads as W
from oracle import grkv_carrier_oracle as CO
from oracle import grkv_oracle as O
from tests.parity import to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _run(cfg, q, K, V):
    import paper_2605_31105_amd as G
    qd, Kd, Vd = (to_device(a, cfg.dtype) for a in (q, K, V))
    res = G.compress(qd, Kd, Vd, cfg.window, cfg.budget, cfg.pool_kernel, cfg.lam)
    assign, counts, metrics, lc = G.carrier_stats(Kd, res.idx, cfg.group, res.stats)
    torch.cuda.synchronize()
    return dict(idx=res.idx.cpu().numpy().astype(np.int64), stats=res.stats.cpu().numpy(),
                assign=assign.cpu().numpy(), counts=counts.cpu().numpy(),
                metrics=metrics.cpu().numpy(), l_common=float(lc.cpu()[0]))


def _check_unit(cfg, K, gpu, u):
    Kd = W.decode(K[u], cfg.dtype)
    idx = gpu["idx"][u]
    ga = gpu["assign"][u].astype(np.int64)
    oa = CO.carrier_assignment(Kd, idx)
    assert np.array_equal(ga < 0, oa < 0)
    ev = np.flatnonzero(oa >= 0)
    diff = ev[ga[ev] != oa[ev]]
    if diff.size:
        Cm = CO.cosine_matrix(Kd[diff], Kd[idx])
        best = Cm.max(axis=1)
        chosen = Cm[np.arange(diff.size), ga[diff]]
        assert np.all(chosen >= best - 1e-5), "unit %d: a non-tie assignment differs" % u
    # metrics of the GPU's assignment, loads exact
    m = CO.carrier_metrics(ga, idx)
    assert np.array_equal(gpu["counts"][u], m["counts"])
    want = [m[k] for k in ("b", "b_eff", "a_max", "gini", "boundary_fraction", "boundary_share",
                           "enrichment", "boundary_interior_load")]
    np.testing.assert_allclose(gpu["metrics"][u], np.array(want, dtype=np.float64), rtol=2e-6,
                               equal_nan=True)
    return dict(unit=u, evicted=int(ev.size), differ=int(diff.size),
                b_over_c=m["b"] / idx.size, beff_over_c=m["b_eff"] / idx.size,
                a_max=m["a_max"], enrichment=m["enrichment"])


def _lcommon_check(gpu):
    st = gpu["stats"].astype(np.float64)
    want = float(np.sum(st[:, 2] * st[:, 0]) / np.sum(st[:, 0]))
    assert abs(gpu["l_common"] - want) <= 1e-6 * max(want, 1e-30)


def test_carrier_config2():
    cfg = W.config(2)
    q, K, V = W.make_batch(cfg)
    gpu = _run(cfg, q, K, V)
    for u in range(cfg.units):
        print(_check_unit(cfg, K, gpu, u), flush=True)
    _lcommon_check(gpu)
    # L_common against the oracle's own value step on these units
    yf, yc = [], []
    for u in range(cfg.units):
        r = O.compress_unit(*(W.decode(a[u], cfg.dtype) for a in (q, K, V)), cfg.window,
                            cfg.budget, cfg.pool_kernel, cfg.lam)
        yf.append(r["Y"])
        yc.append(r["X"] @ r["Vstar"])
    want = CO.l_common(yf, yc)
    assert abs(gpu["l_common"] - want) <= 2e-3 * want, (gpu["l_common"], want)


@pytest.mark.parametrize("label,over", [
    ("head-dim-64", dict(head_dim=64)),
    ("ragged-n", dict(n=1000, budget=200)),
    ("budget-eq-n", dict(n=640, budget=640)),
    ("budget-eq-window", dict(budget=32)),
], ids=["head-dim-64", "ragged-n", "budget-eq-n", "budget-eq-window"])
def test_carrier_edges(label, over):
    base = dict(layers=1, kv_heads=2, n=2048, budget=256)
    base.update(over)
    cfg = W.config(2, **base)
    q, K, V = W.make_batch(cfg)
    gpu = _run(cfg, q, K, V)
    for u in range(cfg.units):
        print(label, _check_unit(cfg, K, gpu, u), flush=True)
    if label == "budget-eq-n":
        assert np.all(gpu["assign"] == -1) and np.all(gpu["metrics"][:, 0] == 0)


def test_carrier_config4_sampled():
    cfg = W.config(4)
    q, K, V = W.make_batch(cfg)
    gpu = _run(cfg, q, K, V)
    for u in (0, 255):
        print(_check_unit(cfg, K, gpu, u), flush=True)
    _lcommon_check(gpu)
    # every unit: loads sum to the evicted count, b <= c, b_eff <= b
    c = cfg.budget
    assert np.all(gpu["counts"].sum(axis=1) == cfg.n - c)
    met = gpu["metrics"]
    assert np.all(met[:, 0] <= c) and np.all(met[:, 1] <= met[:, 0] + 1e-3)
