"""GPU parity of the budget front-ends: adaptive per-head budgets (exact
integers from the GPU's pooled scores) and ragged per-unit compression (every
unit against the float64 oracle with its own budget, to the parity bar of the
uniform path)."""
import numpy as np
import pytest

import workloads as W
from oracle import grkv_frontend_oracle as FO
from oracle import grkv_oracle as O
from tests.parity import D_TOL, V_TOL, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _pooled(cfg, qd, Kd, Vd):
    import paper_2605_31105_amd as G
    res = G.compress(qd, Kd, Vd, cfg.window, cfg.budget, cfg.pool_kernel, cfg.lam)
    return G.intermediates(res)["pooled"].contiguous()


@pytest.mark.parametrize("cfg_id", [2, 4])
def test_adaptive_budgets(cfg_id):
    import paper_2605_31105_amd as G
    cfg = W.config(cfg_id)
    q, K, V = W.make_batch(cfg)
    qd, Kd, Vd = (to_device(a, cfg.dtype) for a in (q, K, V))
    pooled = _pooled(cfg, qd, Kd, Vd)
    got = G.adaptive_budgets(pooled, cfg.layers, cfg.kv_heads, cfg.budget, cfg.window)
    torch.cuda.synchronize()
    got = got.cpu().numpy()
    want = FO.adaptive_budgets(pooled.cpu().numpy().astype(np.float64), cfg.layers,
                               cfg.kv_heads, cfg.budget, cfg.window)
    print("budgets", got[:16], flush=True)
    assert np.array_equal(got, want)
    assert np.all(got.reshape(cfg.layers, cfg.kv_heads).sum(axis=1) == cfg.kv_heads * cfg.budget)


def _ragged_check(cfg, q, K, V, budgets, units=None, **opts):
    """Every unit (or the sampled ``units``) against the oracle with its own
    budget; every unit's retained set checked for the properties that hold at
    any size."""
    import paper_2605_31105_amd as G
    qd, Kd, Vd = (to_device(a, cfg.dtype) for a in (q, K, V))
    idx, k_out, v_out, stats, off = G.compress_ragged(qd, Kd, Vd, cfg.window, budgets,
                                                      cfg.pool_kernel, cfg.lam, **opts)
    torch.cuda.synchronize()
    idx, v_out, stats = idx.cpu().numpy(), v_out.cpu().numpy(), stats.cpu().numpy()
    kc = k_out.cpu()
    kb = kc.view(torch.int16).numpy().view(np.uint16) if cfg.dtype == "bf16" else kc.numpy()
    oo = {k: v for k, v in opts.items() if k in ("n_sink", "beta", "fix_window", "causal_window")}
    opt = O.Options(**oo) if oo else None
    assert np.array_equal(off, FO.packed_offsets(budgets))
    for u, b in enumerate(budgets):
        ids = idx[int(off[u]):int(off[u]) + int(b)]
        assert np.all(np.diff(ids) > 0)
        assert np.array_equal(ids[-cfg.window:], np.arange(cfg.n - cfg.window, cfg.n))
    assert np.all(stats[:, 3] == 0)
    for u in (range(len(budgets)) if units is None else units):
        b = int(budgets[u])
        s = slice(int(off[u]), int(off[u]) + b)
        r = O.compress_unit(*(W.decode(a[u], cfg.dtype) for a in (q, K, V)), cfg.window, b,
                            cfg.pool_kernel, cfg.lam, opt)
        assert np.array_equal(idx[s], r["idx"]), "unit %d: retained set" % u
        assert np.array_equal(kb[s], K[u][r["idx"]])
        verr = np.abs(v_out[s] - r["Vstar"]).max() / np.abs(r["Vstar"]).max()
        print(dict(unit=u, budget=b, v_err=float(verr), d=float(stats[u, 2]),
                   d_oracle=float(r["D_after"])), flush=True)
        assert verr <= V_TOL and stats[u, 3] == r["status"]
        if r["D_after"] > 1e-12:
            assert abs(stats[u, 2] - r["D_after"]) / r["D_after"] <= D_TOL
        else:   # budget = n: nothing evicted, the merge is exact
            assert stats[u, 2] <= 1e-6


def test_ragged_pyramid():
    import paper_2605_31105_amd as G
    cfg = W.config(2, layers=4, kv_heads=2, n=2048, budget=256)
    q, K, V = W.make_batch(cfg)
    budgets = G.pyramid_budgets(cfg.layers, cfg.kv_heads, cfg.budget, cfg.window, cfg.n)
    assert len(set(budgets.tolist())) == cfg.layers
    _ragged_check(cfg, q, K, V, budgets)


def test_ragged_adaptive():
    import paper_2605_31105_amd as G
    cfg = W.config(2)
    q, K, V = W.make_batch(cfg)
    qd, Kd, Vd = (to_device(a, cfg.dtype) for a in (q, K, V))
    budgets = G.adaptive_budgets(_pooled(cfg, qd, Kd, Vd), cfg.layers, cfg.kv_heads, cfg.budget,
                                 cfg.window).cpu().numpy()
    _ragged_check(cfg, q, K, V, budgets)


def test_ragged_token_based_and_mixed_budgets():
    # pool width 1 (token-based scoring), budgets differing unit to unit
    cfg = W.config(2, layers=1, kv_heads=4, n=1000, budget=200, pool_kernel=1)
    q, K, V = W.make_batch(cfg)
    _ragged_check(cfg, q, K, V, [200, 32, 1000, 137])


def test_ragged_uniform_equals_compress():
    import paper_2605_31105_amd as G
    cfg = W.config(2)
    q, K, V = W.make_batch(cfg)
    qd, Kd, Vd = (to_device(a, cfg.dtype) for a in (q, K, V))
    a = G.compress(qd, Kd, Vd, cfg.window, cfg.budget, cfg.pool_kernel, cfg.lam)
    idx, k_out, v_out, stats, _ = G.compress_ragged(qd, Kd, Vd, cfg.window,
                                                    [cfg.budget] * cfg.units, cfg.pool_kernel,
                                                    cfg.lam)
    torch.cuda.synchronize()
    assert torch.equal(a.idx.reshape(-1), idx) and torch.equal(a.k_out.reshape(-1, cfg.head_dim), k_out)
    assert torch.equal(a.v_out.reshape(-1, cfg.head_dim), v_out) and torch.equal(a.stats, stats)


def test_ragged_full_workload_pyramid_and_adaptive_sampled():
    # the 32-layer n=32k workload in one ragged call per front-end, sampled
    # units against the oracle (the adaptive sample holds the smallest and
    # the largest budget)
    import paper_2605_31105_amd as G
    cfg = W.config(4)
    q, K, V = W.make_batch(cfg)
    b = G.pyramid_budgets(cfg.layers, cfg.kv_heads, cfg.budget, cfg.window, cfg.n)
    _ragged_check(cfg, q, K, V, b, units=(0, 37, 128, 255))
    qd, Kd, Vd = (to_device(a, cfg.dtype) for a in (q, K, V))
    b = G.adaptive_budgets(_pooled(cfg, qd, Kd, Vd), cfg.layers, cfg.kv_heads, cfg.budget,
                           cfg.window).cpu().numpy()
    del qd, Kd, Vd
    _ragged_check(cfg, q, K, V, b, units=(int(np.argmin(b)), int(np.argmax(b)), 101, 200))


@pytest.mark.parametrize("label,cfg_id,over,budgets", [
    ("fp32", 1, {}, [16, 300]),
    ("bf16-m256", 2, dict(layers=1, kv_heads=2, n=2048, window=64, budget=512), [512, 300]),
], ids=["fp32", "bf16-m256"])
def test_ragged_generic_path(label, cfg_id, over, budgets):
    # shapes outside the bf16 fast path run one call per run of equal budgets
    cfg = W.config(cfg_id, **over)
    q, K, V = W.make_batch(cfg)
    _ragged_check(cfg, q, K, V, budgets)
